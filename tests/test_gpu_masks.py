"""GPU: the action masks of the benchmark's route kernels under host-side
model changes. In the c2, c3 and c4 shapes (the 64-row persistent kernel at a
grid small enough that a tick is heavy, and the streaming kernel), models are
disabled or given no slots in a third of the envs for a span of ticks, then
restored. A row's valid actions come from the validity bytes of its env's
snapshot row (rewritten by the host calls), so within the span no action may
name such a model; the lockstep with the oracle checks every action and the
integer state on every tick."""
import numpy as np
import pytest

import workload
from gpu_util import Pair, note

pytestmark = pytest.mark.gpu

CASES = [("c2", dict(E=64, lam=64.0)), ("c4", dict(E=96)), ("c3", dict(E=48))]


@pytest.mark.parametrize("name,over", CASES, ids=[c[0] for c in CASES])
def test_masks_follow_host_knobs(name, over):
    cfg = workload.configs.get(name, T=12, **over)
    E, M, K = cfg["E"], cfg["M"], cfg["K"]
    note(f"[masks] {name}: E={E} M={M} K={K}")
    p = Pair(cfg, seed=71, Q=2048)
    p.gpu.set_launch(4, 4)   # four route blocks: every tick is a heavy one
    rng = np.random.default_rng(5)
    off = {}
    for t in range(cfg["T"]):
        if t == 3:
            for e in range(0, E, 3):
                ms = rng.choice(M, size=1 + e % (M - 1), replace=False)
                for m in ms:
                    if (e + int(m)) % 2:
                        p.gpu.set_enabled(e, int(m), 0)
                        p.orc.set_enabled(e, int(m), 0)
                    else:
                        p.gpu.set_capacity(e, int(m), 0)
                        p.orc.set_capacity(e, int(m), 0)
                off[e] = {int(m) for m in ms}
        if t == 8:
            caps = workload.gen.capacities(cfg, 71)
            for e, ms in off.items():
                for m in ms:
                    p.gpu.set_enabled(e, m, 1)
                    p.orc.set_enabled(e, m, 1)
                    p.gpu.set_capacity(e, m, int(caps[e, m]))
                    p.orc.set_capacity(e, m, int(caps[e, m]))
        arr = p.arrivals(t)
        act = p.step(arr, mode="tick" if t % 2 else "route+schedule")
        if 3 <= t < 8:
            o = arr["offsets"]
            for e, ms in off.items():
                a = act[o[e]:o[e + 1]]
                a = a[a >= 0]
                assert not np.isin(a // K, list(ms)).any(), (name, t, e, sorted(ms))
        p.compare_state(ctx=f"{name} t={t}")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()
