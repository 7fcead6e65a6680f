"""GPU parity of the blackbox congestion proxy (Sec. 5.5, App. C) through
im_set_rpm_limit: the whole integer state, including the 60-tick dispatch
history and count, bit-exact with the oracle, and the logits (whose
queue-depth feature becomes recent dispatches / limit) within the tolerance.
Cases: the closed-form burst (5 dispatches per 60-tick window), random
workloads with mixed limits and a limit changed mid-run, an env skipped for
bad input (its window still slides), and checkpoint/resume of the window."""
import numpy as np
import pytest

import workload
from gpu_util import Pair, need_gpu, note
from helpers import assert_state_equal, tiny_cfg

pytestmark = pytest.mark.gpu


def _set(p, e, m, r):
    p.gpu.set_rpm_limit(e, m, r)
    p.orc.set_rpm_limit(e - p.e0, m, r)


def test_rpm_burst_closed_form():
    need_gpu()
    cfg = tiny_cfg(M=1, K=1, widths=[32, 1], key_mode="fcfs", qcap=128, cap_hi=8,
                   max_arrivals=128, budget_hi=1000, T=150)
    note("[rpm_burst]")
    p = Pair(cfg, seed=1, Q=4)
    _set(p, 0, 0, 5)
    z = np.zeros(0, np.int32)
    empty = dict(offsets=np.array([0, 0], np.int32), q_idx=z, budget=z.astype(np.int16),
                 base_svc=z.astype(np.int16))
    burst = dict(offsets=np.array([0, 100], np.int32), q_idx=np.zeros(100, np.int32),
                 budget=np.full(100, 1000, np.int16), base_svc=np.full(100, 10, np.int16))
    for t in range(cfg["T"]):
        p.step(burst if t == 0 else empty)
        if t % 10 == 0 or t % 60 in (59, 0, 1):
            s = p.compare_state(ctx=f"burst t={t}")
            assert s["started"][0, 0] == 5 * (t // 60 + 1)
    p.close()


@pytest.mark.parametrize("name,E,T", [("c0", 1, 150), ("c2", 6, 90), ("c4", 8, 70)])
def test_rpm_mixed_limits(name, E, T):
    need_gpu()
    cfg = workload.configs.get(name, E=E, T=T)
    note(f"[rpm_mixed] {name} E={E} T={T}")
    p = Pair(cfg, seed=41, Q=256)
    rng = np.random.default_rng(5)
    for e in range(E):
        for m in range(cfg["M"]):
            if rng.random() < 0.5:
                _set(p, e, m, int(rng.integers(1, 40)))
    for t in range(T):
        if t == T // 2:
            _set(p, 0, 0, 2)                    # a limit changed mid-run
            _set(p, E - 1, cfg["M"] - 1, 0)     # and one model made white-box again
        p.step(p.arrivals(t))
        if t % 10 == 9:
            p.compare_state(ctx=f"{name} t={t}")
    assert p.gpu.error() == 0
    p.close()


def test_rpm_window_slides_in_a_skipped_env():
    torch = need_gpu()
    cfg = workload.configs.get("c0", T=80, lam=8.0)
    note("[rpm_skipped_env]")
    p = Pair(cfg, seed=42, Q=64)
    for m in range(cfg["M"]):
        _set(p, 0, m, 4)
    for t in range(cfg["T"]):
        arr = p.arrivals(t)
        if t in (20, 61) and arr["q_idx"].size:
            arr = dict(arr, budget=arr["budget"].copy())
            arr["budget"][0] = 0                # invalid: the env is skipped this tick
            p.step(arr, check_logits=False)
            p.gpu.clear_error()
            p.orc.clear_error()
        else:
            p.step(arr)
        if t % 8 == 7 or t in (20, 21, 61, 62):
            p.compare_state(ctx=f"t={t}")
    p.close()


def test_rpm_checkpoint_resume():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2", E=10, T=90, lam=16.0)
    note("[rpm_checkpoint]")
    a = Pair(cfg, seed=43, Q=256)
    for e in range(cfg["E"]):
        _set(a, e, e % cfg["M"], 3 + e)
    for t in range(70):
        a.step(a.arrivals(t), mode="tick")
    snap = a.gpu.state()
    assert snap["rpm_hist"].sum() > 0
    b = Pair(cfg, seed=43, Q=256)
    b.gpu.write_state(0, snap)
    assert_state_equal(b.gpu.state(), snap, ctx="round trip")
    for t in range(70, 90):
        arr = a.arrivals(t)
        dev = P.device_arrivals(arr)
        for q in (a, b):
            act = torch.zeros(max(len(arr["q_idx"]), 1), dtype=torch.int32, device="cuda")
            q.gpu.tick(dev, act)
    assert_state_equal(a.gpu.state(), b.gpu.state(), ctx="resume")
    a.close()
    b.close()
