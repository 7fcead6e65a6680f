"""GPU parity: the HIP library against the oracle, element by element.

Lockstep per tick: logits within the tolerance (1e-4 fp32, 2e-2 bf16, relative
to the row's largest oracle logit), actions equal except at near ties (the
oracle then adopts the GPU's action), and the whole integer state bit-exact.
Small sizes compare every env every tick; full sizes run the benchmark's
launch configuration (im_tick over all envs) and compare a sampled subset of
envs, which is exact because envs are independent."""
import numpy as np
import pytest

import workload
from gpu_util import Pair, note

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,E,T", [("c0", 1, 100), ("c1", 12, 40), ("c2", 12, 40),
                                      ("c3", 4, 30), ("c4", 16, 40)])
def test_lockstep_small(name, E, T):
    cfg = workload.configs.get(name, E=E, T=T)
    note(f"[lockstep_small] {name} E={E} T={T}")
    p = Pair(cfg, seed=11, Q=512)
    for t in range(T):
        p.step(p.arrivals(t))
        p.compare_state(ctx=f"{name} t={t}")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()


@pytest.mark.parametrize("name,lam", [("c2", 4.0), ("c2", 16.0)])
def test_lockstep_load_sweep(name, lam):
    cfg = workload.configs.get(name, E=16, T=60, lam=lam)
    note(f"[load_sweep] {name} lam={lam}")
    p = Pair(cfg, seed=12, Q=512)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
    p.compare_state(ctx=f"{name} lam={lam}")
    p.close()


@pytest.mark.parametrize("mode", ["deadline", "fcfs"])
def test_lockstep_key_modes(mode):
    cfg = workload.configs.get("c1", E=8, T=40, key_mode=mode)
    note(f"[key_modes] {mode}")
    p = Pair(cfg, seed=13, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 8 == 7:
            p.compare_state(ctx=f"{mode} t={t}")
    p.close()


# Full sizes in the benchmark's launch configuration (im_tick over all envs);
# the oracle follows a sampled, contiguous block of envs. Every run covers the
# whole workload: c2 and c3 reach pools of about 2,000 (c2) and 1,000 (c3,
# M = 16) entries whose fronts drain and are refilled, c4 saturates its
# 512-entry queues from about tick 40 on (tail drops every tick).
FULL = [("c1", dict(), 0, 8), ("c2", dict(lam=64.0), 1000, 1006),
        ("c3", dict(), 2048, 2052), ("c4", dict(), 65530, 65536)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,over,e0,e1", FULL)
def test_full_size_sampled(name, over, e0, e1):
    cfg = workload.configs.get(name, **over)
    note(f"[full_size] {name} E={cfg['E']} T={cfg['T']} envs [{e0},{e1})")
    p = Pair(cfg, seed=0, e0=e0, e1=e1)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t), mode="tick")
        if t % 32 == 31:
            p.compare_state(ctx=f"{name} t={t}")
            note(f"  t={t} ok")
    p.compare_state(ctx=f"{name} end")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()
