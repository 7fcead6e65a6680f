"""GPU parity on policy shapes outside the five workloads, so that every
route kernel variant runs: fp32 with one wave per 16-row tile (hidden width 32)
and feature-split (hidden widths in tile quads), fp32 and bf16 with several
output tiles, and the generic (non-persistent) bf16 kernel. Lockstep with the
oracle as in the workload tests (logits within 1e-4 fp32 / 2e-2 bf16 of the
row's largest oracle logit, actions equal except at near ties, integer state
bit-exact), greedy route and schedule, then RL outputs with a value head."""
import pytest

import workload
from gpu_util import Pair, note

pytestmark = pytest.mark.gpu

# (id, base workload, overrides); feat_dim covers [emb | 4M stats | budget]
SHAPES = [
    ("f32_h32_3layer", "c1", dict(widths=[32, 32, 15])),
    ("f32_h128_2layer_24act", "c1", dict(M=8, K=3, feat_dim=98, widths=[128, 24])),
    ("f32_h64_3layer_64act", "c1", dict(M=16, K=4, feat_dim=130, widths=[64, 64, 64])),
    ("bf16_h128_3layer", "c2", dict(widths=[128, 128, 15])),
    ("bf16_h64_2layer_64act", "c2", dict(M=16, K=4, feat_dim=130, widths=[64, 64])),
    # 40 zero features past [emb | 4M stats | budget]: the vector gather must not read the
    # snapshot row past the load statistics
    ("bf16_h256_3layer_feat_pad40", "c2", dict(feat_dim=64 + 4 * 5 + 1 + 40)),
]


@pytest.mark.parametrize("sid,base,over", SHAPES, ids=[s[0] for s in SHAPES])
def test_shape_lockstep(sid, base, over):
    cfg = workload.configs.get(base, E=10, T=30, lam=24.0, **over)
    note(f"[shape_lockstep] {sid}")
    p = Pair(cfg, seed=31, Q=512)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 6 == 5:
            p.compare_state(ctx=f"{sid} t={t}")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()


# with a value head: the pool's last layer gets one more row (M*K + 1 outputs)
RL_SHAPES = [
    ("f32_h128_2layer_24act_value", "c1", dict(M=8, K=3, feat_dim=98, widths=[128, 24])),
    ("f32_h32_3layer_value", "c1", dict(widths=[32, 32, 15])),
    ("bf16_h128_3layer_value", "c2", dict(widths=[128, 128, 15])),
]


@pytest.mark.parametrize("sid,base,over", RL_SHAPES, ids=[s[0] for s in RL_SHAPES])
def test_shape_rl_lockstep(sid, base, over):
    cfg = workload.configs.get(base, E=8, T=20, lam=24.0, value_head=True, **over)
    note(f"[shape_rl_lockstep] {sid}")
    p = Pair(cfg, seed=32, Q=512)
    for t in range(cfg["T"]):
        p.step_rl(p.arrivals(t), seed=0x5EED1000 + t)
        if t % 5 == 4:
            p.compare_state(ctx=f"{sid} t={t}")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()
