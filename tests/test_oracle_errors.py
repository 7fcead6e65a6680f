"""Oracle error rules: an env whose tick input is invalid is left untouched
(no counters, no id advance, no service) and the error bits are raised;
other envs proceed normally."""
import numpy as np
import pytest

import oracle
import workload
from helpers import assert_state_equal, make_oracle


def _run(cfg, seed, T, Q):
    o, _ = make_oracle(cfg, seed=seed, Q=Q)
    cnt = workload.gen.counts(cfg, seed)
    for t in range(T):
        o.tick(workload.gen.tick(cfg, seed, t, cnt[t], Q))
    return o, cnt


@pytest.mark.parametrize("what,bit", [("q_idx", oracle.ERR_QIDX), ("budget", oracle.ERR_BUDGET),
                                      ("base_svc", oracle.ERR_SVC), ("action", oracle.ERR_ACTION),
                                      ("count", oracle.ERR_COUNT)])
def test_invalid_env_untouched(what, bit):
    cfg = workload.configs.get("c1", E=3, T=12, max_arrivals=40)
    Q = 64
    o, cnt = _run(cfg, 9, 10, Q)
    arr = workload.gen.tick(cfg, 9, 10, cnt[10], Q)
    before = o.state()
    act, _ = o.route(arr)
    o.clear_error()
    lo, hi = arr["offsets"][1], arr["offsets"][2]
    assert hi > lo
    if what == "q_idx":
        arr["q_idx"][lo] = Q
    elif what == "budget":
        arr["budget"][lo] = 0
    elif what == "base_svc":
        arr["base_svc"][lo] = 0
    elif what == "action":
        act[lo] = cfg["A"]
    elif what == "count":
        cfg2 = dict(cfg)
        extra = 41 - (hi - lo)
        n = len(arr["q_idx"])
        for k in ("q_idx", "budget", "base_svc"):
            arr[k] = np.insert(arr[k], hi, np.repeat(arr[k][lo:lo + 1], extra))
        act = np.insert(act, hi, np.zeros(extra, np.int32))
        arr["offsets"] = arr["offsets"].copy()
        arr["offsets"][2:] += extra
    o.schedule(arr, act)
    assert o.error & bit
    after = o.state()
    sel = np.array([1])
    for k in ("next_id", "arrived", "rej_nomodel", "qlen", "busy", "completed", "hist", "slots"):
        assert np.array_equal(np.asarray(before[k])[sel], np.asarray(after[k])[sel]), k
    assert after["arrived"][0] > before["arrived"][0] or cnt[10][0] == 0


def test_route_marks_bad_qidx_rows():
    cfg = workload.configs.get("c0")
    o, _ = make_oracle(cfg, seed=1, Q=16)
    arr = dict(offsets=np.array([0, 3], np.int32), q_idx=np.array([0, 16, -1], np.int32),
               budget=np.array([5, 5, 5], np.int16), base_svc=np.array([1, 1, 1], np.int16))
    act, lg = o.route(arr)
    assert act[1] == -1 and act[2] == -1 and act[0] >= 0
    assert np.all(lg[1:] == 0.0)
    assert o.error & oracle.ERR_QIDX
