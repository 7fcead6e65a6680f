"""Oracle of the blackbox congestion proxy (Sec. 5.5, App. C) pinned to
closed forms and invariants.

A model with an RPM limit R dispatches (fills a service slot) only while fewer
than R dispatches fall in the last 60 ticks; its queue-depth feature becomes
recent dispatches / R. Pins: a burst of 100 requests to one model with 8
slots, R = 5 and 10-tick services is dispatched exactly 5 per 60-tick window
(started after tick t = 5 (floor(t / 60) + 1)), the feature equals the window
count times the fp32 reciprocal of R, and on a random workload with mixed
limits no 60-tick window ever holds more than R dispatches while white-box
models are unaffected."""
import numpy as np

import oracle
import workload
from helpers import make_oracle, tiny_cfg


def _burst(n):
    return dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32),
                budget=np.full(n, 1000, np.int16), base_svc=np.full(n, 10, np.int16))


def _empty():
    z = np.zeros(0, np.int32)
    return dict(offsets=np.array([0, 0], np.int32), q_idx=z, budget=z.astype(np.int16),
                base_svc=z.astype(np.int16))


def test_rate_limited_dispatch_closed_form():
    cfg = tiny_cfg(M=1, K=1, widths=[32, 1], key_mode="fcfs", qcap=128, cap_hi=8,
                   max_arrivals=128, budget_hi=1000)
    o, _ = make_oracle(cfg, seed=1, Q=4, cap=np.full((1, 1), 8, np.int32))
    o.set_rpm_limit(0, 0, 5)
    inv = float(np.float32(1.0 / 5))
    for t in range(300):
        x = o.features(0, 0, 10)
        s = o.state()
        assert x[cfg["embed_dim"]] == float(np.float32(s["rpm_count"][0, 0]) * np.float32(inv))
        o.tick(_burst(100) if t == 0 else _empty())
        s = o.state()
        assert s["started"][0, 0] == 5 * (t // 60 + 1), t
        assert s["rpm_count"][0, 0] == 5          # 5 dispatches at the window's first tick
        assert int(s["rpm_hist"][0, 0].sum()) == s["rpm_count"][0, 0] <= 5


def test_window_never_exceeds_limit():
    cfg = workload.configs.get("c0", T=200, lam=6.0)
    o, _ = make_oracle(cfg, seed=3, Q=32)
    limits = [3, 0, 12, 0, 1]
    for m, r in enumerate(limits):
        o.set_rpm_limit(0, m, r)
    cnt = workload.gen.counts(cfg, 3)
    started_hist = []
    for t in range(cfg["T"]):
        o.tick(workload.gen.tick(cfg, 3, t, cnt[t], 32))
        s = o.state()
        started_hist.append(s["started"][0].copy())
        assert np.array_equal(s["rpm_hist"][0].sum(axis=1), s["rpm_count"][0])
    st = np.array(started_hist)
    per_tick = np.diff(np.vstack([np.zeros(cfg["M"], np.int64), st]), axis=0)
    for m, r in enumerate(limits):
        if r == 0:
            continue
        win = np.convolve(per_tick[:, m], np.ones(60, np.int64))[:len(per_tick)]
        assert win.max() <= r, (m, win.max(), r)
        assert win.max() == r           # the load saturates every limited model


def test_zero_limit_is_whitebox():
    cfg = workload.configs.get("c2", E=3, T=40)
    a, _ = make_oracle(cfg, seed=4, Q=64)
    b, _ = make_oracle(cfg, seed=4, Q=64)
    for m in range(cfg["M"]):
        b.set_rpm_limit(1, m, 0)
    cnt = workload.gen.counts(cfg, 4)
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 4, t, cnt[t], 64)
        a.tick(arr)
        b.tick(arr)
    sa, sb = a.state(), b.state()
    for k in ("qlen", "started", "completed", "queues", "slots", "lat_sum"):
        np.testing.assert_array_equal(sa[k], sb[k])
