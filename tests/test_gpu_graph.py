"""Ticks captured into a HIP graph: replaying the graph must give exactly the
state of the same ticks launched eagerly. The tick counter lives in device
memory, so a replayed tick advances time; the graph's arrival buffers are
refilled between replays (a fixed batch size, as rollouts use)."""
import numpy as np
import pytest

import workload
from gpu_util import Pair, need_gpu, note
from helpers import assert_state_equal

pytestmark = pytest.mark.gpu


def _fixed_total_tick(cfg, rng, n, Q):
    E = cfg["E"]
    counts = rng.multinomial(n, np.ones(E) / E).astype(np.int32)
    counts = np.minimum(counts, cfg["max_arrivals"])
    counts[0] += n - counts.sum()
    off = np.zeros(E + 1, np.int32)
    off[1:] = np.cumsum(counts)
    return dict(offsets=off, q_idx=rng.integers(0, Q, n).astype(np.int32),
                budget=rng.integers(cfg["budget_lo"], cfg["budget_hi"] + 1, n).astype(np.int16),
                base_svc=rng.integers(1, 9, n).astype(np.int16))


@pytest.mark.parametrize("name", ["c2", "c4"])
def test_graph_replays_match_eager(name):
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get(name, E=64, T=24)
    note(f"[graph] {name}")
    Q = 256
    eager = Pair(cfg, seed=31, Q=Q, e0=0, e1=1)
    graphed = Pair(cfg, seed=31, Q=Q, e0=0, e1=1)
    rng = np.random.default_rng(3)
    n = cfg["E"] * 8
    buf = {k: torch.zeros(cfg["E"] + 1 if k == "offsets" else n,
                          dtype=torch.int32 if k in ("offsets", "q_idx") else torch.int16,
                          device="cuda") for k in ("offsets", "q_idx", "budget", "base_svc")}
    arr_dev = P.make_arrivals(buf["offsets"], buf["q_idx"], buf["budget"], buf["base_svc"])
    act_g = torch.zeros(n, dtype=torch.int32, device="cuda")
    first = _fixed_total_tick(cfg, rng, n, Q)
    for k in buf:
        buf[k].copy_(torch.from_numpy(first[k]))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        graphed.gpu.tick(arr_dev, act_g)
    torch.cuda.synchronize()
    ticks = [first] + [_fixed_total_tick(cfg, rng, n, Q) for _ in range(cfg["T"] - 1)]
    for t, tk in enumerate(ticks):
        if t > 0:
            for k in buf:
                buf[k].copy_(torch.from_numpy(tk[k]))
        g.replay()
        torch.cuda.synchronize()
        eager.gpu.tick(P.device_arrivals(tk))
        assert_state_equal(graphed.gpu.state(), eager.gpu.state(), ctx=f"{name} replay {t}")
    assert graphed.gpu.state()["t"] == cfg["T"]
    eager.close()
    graphed.close()
