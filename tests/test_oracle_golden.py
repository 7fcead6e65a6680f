"""Oracle pinned to a hand-derived six-tick example (tests/golden/golden_6tick.json).

The paper prints no worked example of the tick, so the fixture was derived by
hand from the rules it states: action decode (Sec. 3), deadline-ordered
per-model queues (Sec. 4.3), bounded concurrency (Table 5) and an EMA latency
signal (Sec. 5.4), with the documented readings for what it leaves open."""
import json
import os

import numpy as np
import pytest

import oracle
import workload

HERE = os.path.dirname(os.path.abspath(__file__))


def golden():
    with open(os.path.join(HERE, "golden", "golden_6tick.json")) as f:
        return json.load(f)


def make_pool(g):
    s = g["setup"]
    A = s["M"] * s["K"]
    cfg = workload.configs.finish(dict(
        index=0, E=1, M=s["M"], K=s["K"], qcap=s["qcap"], cap_lo=1, cap_hi=s["max_slots"],
        budget_lo=1, budget_hi=s["budget_max"], embed_dim=s["embed_dim"],
        feat_dim=s["embed_dim"] + 4 * s["M"] + 1, widths=[A], dtype="f32",
        key_mode=s["key_mode"], max_arrivals=16, lam=1.0, T=6, svc_mu=1.0, svc_sigma=0.5))
    W = [np.zeros((A, cfg["feat_dim"]), np.float32)]
    b = [np.zeros(A, np.float32)]
    emb = np.zeros((4, s["embed_dim"]), np.float32)
    cap = np.array([s["cap"]], np.int32)
    return cfg, oracle.Oracle(cfg, W, b, emb, cap)


def arrivals(tick):
    n = len(tick["arrivals"])
    return dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32),
                budget=np.array([a[0] for a in tick["arrivals"]], np.int16),
                base_svc=np.array([a[1] for a in tick["arrivals"]], np.int16)), \
        np.array([a[2] for a in tick["arrivals"]], np.int32)


def test_golden_six_ticks():
    g = golden()
    cfg, o = make_pool(g)
    for tick in g["ticks"]:
        assert o.t == tick["t"]
        arr, act = arrivals(tick)
        if "features_before" in tick:
            fb = tick["features_before"]
            x = o.features(0, 0, fb["budget"])
            M, Ed = cfg["M"], cfg["embed_dim"]
            for si, row in enumerate(fb["stats"]):
                for m, v in enumerate(row):
                    assert x[Ed + si * M + m] == pytest.approx(v, rel=1e-6, abs=1e-9), (si, m)
            assert x[Ed + 4 * M] == pytest.approx(fb["budget_feature"], rel=1e-6)
        o.schedule(arr, act)
        st = o.state()
        for m in range(cfg["M"]):
            q = st["queues"][0, m, :st["qlen"][0, m]].tolist()
            assert q == tick["queues_after"][m], (tick["t"], m)
            assert st["slots"][0, m, 0].tolist() == tick["slots_after"][m], (tick["t"], m)
        assert st["backlog"][0].tolist() == tick["backlog_after"]
        assert st["ewma"][0].tolist() == tick["ewma_after"]
    st = o.state()
    fin = g["final"]
    assert st["arrived"][0] == fin["arrived"]
    assert st["rej_nomodel"][0] == fin["rej_nomodel"]
    for k, v in fin["per_model"].items():
        assert st[k][0].tolist() == v, k
    for k, v in fin["totals"].items():
        assert int(st[k][0].sum()) == v, k
    assert st["hist"][0].tolist() == fin["hist"]
    assert o.error == 0


def test_golden_mask_at_t2():
    """At t2 model 0's queue is full (qlen == QCAP): routing must avoid it.
    With all-zero weights every logit ties, so the lowest valid action wins."""
    g = golden()
    cfg, o = make_pool(g)
    for tick in g["ticks"][:2]:
        arr, act = arrivals(tick)
        o.schedule(arr, act)
    arr, _ = arrivals(g["ticks"][2])
    act, lg = o.route(arr)
    assert act.tolist() == [2]          # model 0 (actions 0, 1) masked
    assert np.all(lg == 0.0)
