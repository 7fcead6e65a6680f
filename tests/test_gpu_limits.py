"""GPU lockstep with the oracle at the library's size limits: a queue of the
largest capacity (16,384 entries) filled by bursts of 4,096 arrivals per
env-tick (64 row chunks, 16 staging rounds of the schedule step) and drained
through 8 one-tick slots, so the front is refilled from pools of up to 256
chunks; 64 (model, slot) lanes in one service pass (8 models x 8 slots, 64
actions); and the widest feature vector (512)."""
import numpy as np
import pytest

from gpu_util import Pair, note
from helpers import tiny_cfg

pytestmark = pytest.mark.gpu


def _burst(E, counts, Q, rng, budget_hi):
    off = np.zeros(E + 1, np.int32)
    off[1:] = np.cumsum(counts)
    n = int(off[-1])
    return dict(offsets=off, q_idx=rng.integers(0, Q, n).astype(np.int32),
                budget=rng.integers(1, budget_hi + 1, n).astype(np.int16),
                base_svc=np.ones(n, np.int16))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("key_mode", ["fcfs", "slack"])
def test_max_queue_capacity(key_mode):
    cfg = tiny_cfg(M=1, K=2, widths=[32, 2], qcap=16384, cap_lo=8, cap_hi=8, max_slots=8, E=2,
                   max_arrivals=4096, key_mode=key_mode, budget_hi=30000, embed_dim=8)
    note(f"[max_queue] {key_mode}")
    p = Pair(cfg, seed=41, Q=512)
    rng = np.random.default_rng(41)
    E = cfg["E"]
    for t in range(40):
        # five ticks of bursts (past the capacity: tail drops), then drain
        counts = np.array([4096, 4000], np.int32) if t < 5 else np.array([3, 0], np.int32)
        p.step(_burst(E, counts, 512, rng, cfg["budget_hi"]), mode="tick" if t % 2 else "route+schedule")
        if t % 5 == 4:
            p.compare_state(ctx=f"{key_mode} t={t}")
    s = p.gpu.state()
    assert s["rej_overflow"].sum() > 0 and s["started"].sum() > 100
    note(f"  rows={p.rows_checked}")
    assert p.gpu.error() == 0
    p.close()


def test_full_service_pass():
    cfg = tiny_cfg(M=8, K=8, widths=[64, 64], qcap=128, cap_lo=8, cap_hi=8, max_slots=8, E=8, lam=48.0, T=25,
                   max_arrivals=256, budget_hi=60, embed_dim=16, dtype="bf16")
    note("[full_service_pass] M=8 x 8 slots")
    p = Pair(cfg, seed=42, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 6 == 5:
            p.compare_state(ctx=f"t={t}")
    p.compare_state(ctx="end")
    assert p.gpu.error() == 0
    p.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_widest_features(dtype):
    cfg = tiny_cfg(M=4, K=3, embed_dim=448, feat_dim=512, widths=[64, 12], qcap=64, cap_hi=3, E=6,
                   lam=20.0, T=12, max_arrivals=128, budget_hi=60, dtype=dtype)
    note(f"[widest_features] {dtype} D_in={cfg['feat_dim']}")
    p = Pair(cfg, seed=43, Q=128)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
    p.compare_state(ctx="end")
    assert p.gpu.error() == 0
    p.close()
