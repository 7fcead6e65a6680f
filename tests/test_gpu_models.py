"""GPU lockstep with the oracle at model counts that stress the schedule
step's per-model lanes: the largest supported count (M = 32: five bits of
model index in the tail-drop ranks, service in two passes of (model, slot)
lanes), counts that are not powers of two, and a chain pool with many models.
Queues are short, so fronts fill, pools take appends and full queues drop
newcomers (the admitted-rows-only sort) within a few ticks."""
import pytest

from gpu_util import Pair, note
from helpers import tiny_cfg

pytestmark = pytest.mark.gpu

CASES = [
    ("m32_f32", dict(M=32, K=2, dtype="f32", widths=[64, 64])),
    ("m32_bf16", dict(M=32, K=2, dtype="bf16", widths=[64, 64])),
    ("m7_bf16", dict(M=7, K=3, dtype="bf16", widths=[64, 21])),
    ("m17_f32", dict(M=17, K=3, dtype="f32", widths=[64, 51])),
    ("m12_chain", dict(M=12, K=2, dtype="bf16", widths=[64, 24], max_steps=3)),
]


@pytest.mark.parametrize("name,over", CASES, ids=[c[0] for c in CASES])
def test_lockstep_model_counts(name, over):
    cfg = tiny_cfg(qcap=48, cap_hi=3, E=20, embed_dim=32, lam=40.0, T=30, max_arrivals=256,
                   budget_hi=80, **over)
    note(f"[model_counts] {name}: M={cfg['M']} K={cfg['K']} A={cfg['A']}")
    p = Pair(cfg, seed=31, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t), mode="tick" if t % 2 else "route+schedule")
        if t % 5 == 4:
            p.compare_state(ctx=f"{name} t={t}")
    p.compare_state(ctx=f"{name} end")
    s = p.gpu.state()
    assert s["rej_overflow"].sum() > 0, "full queues were reached"
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()
