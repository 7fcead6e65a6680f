"""Oracle of the dual update (Eq. 7) pinned to closed forms.

Each completion adds floor(2^16 latency / budget) to a per-model cost counter
(Eq. 2's C_k = l_k / beta in Q16); the update takes the mean cost over the
completions since the previous update. Pins: a single-slot FCFS model fed one
request every 5 ticks serves every request in exactly its service time, so the
cost of each is svc / budget and lambda follows the closed-form ramp down
(C = 1/2) or up to lambda_max (C = 2); with every budget 1 the cost counter is
2^16 times the latency sum; no completion leaves lambda unchanged."""
import numpy as np
import pytest

import workload
from helpers import make_oracle, tiny_cfg


def _one_request(budget, svc):
    return dict(offsets=np.array([0, 1], np.int32), q_idx=np.array([0], np.int32),
                budget=np.array([budget], np.int16), base_svc=np.array([svc], np.int16))


def _empty():
    z = np.zeros(0, np.int32)
    return dict(offsets=np.array([0, 0], np.int32), q_idx=z, budget=z.astype(np.int16),
                base_svc=z.astype(np.int16))


@pytest.mark.parametrize("budget,svc,direction", [(8, 4, -1), (2, 4, +1), (12, 3, -1)])
def test_closed_form_ramp(budget, svc, direction):
    cfg = tiny_cfg(M=1, K=1, widths=[32, 1], key_mode="fcfs", qcap=16, cap_hi=1)
    o, _ = make_oracle(cfg, seed=1, Q=4, cap=np.ones((1, 1), np.int32))
    lam, eta, lmax = 0.2, 0.001, 1.0
    cost = svc / budget
    updates = 0
    for t in range(400):
        arr = _one_request(budget, svc) if t % 5 == 0 else _empty()
        act = o.tick(arr)
        assert np.all(act == 0)
        if t % 10 == 9:
            lam = o.dual_update(lam, eta, lmax)
            updates += 1
            exp = min(max(0.2 + updates * eta * (cost - 1.0), 0.0), lmax)
            assert lam == pytest.approx(exp, abs=1e-12)
    s = o.state()
    n = int(s["completed"][0, 0])
    assert s["lat_sum"][0, 0] == n * svc                      # every request served in svc ticks
    assert s["cost_q16"][0, 0] == n * ((svc << 16) // budget)
    assert (lam < 0.2) if direction < 0 else (lam > 0.2)


def test_unit_budgets_cost_is_scaled_latency():
    cfg = workload.configs.get("c0", T=60, budget_lo=1, budget_hi=1)
    o, _ = make_oracle(cfg, seed=2, Q=32)
    cnt = workload.gen.counts(cfg, 2)
    lam = 0.5
    last_n = last_l = 0
    for t in range(cfg["T"]):
        o.tick(workload.gen.tick(cfg, 2, t, cnt[t], 32))
        if t % 15 == 14:
            s = o.state()
            np.testing.assert_array_equal(s["cost_q16"], s["lat_sum"] << 16)
            n, l = int(s["completed"].sum()), int(s["lat_sum"].sum())
            new = o.dual_update(lam, 0.01, 1.0)
            if n > last_n:
                assert new == pytest.approx(min(max(lam + 0.01 * ((l - last_l) / (n - last_n) - 1), 0), 1),
                                            abs=1e-12)
            last_n, last_l, lam = n, l, new


def test_no_completion_keeps_lambda():
    cfg = tiny_cfg(M=1, K=1, widths=[32, 1])
    o, _ = make_oracle(cfg, seed=3, Q=4)
    for _ in range(3):
        o.tick(_empty())
    assert o.dual_update(0.37, 0.5, 1.0) == 0.37
