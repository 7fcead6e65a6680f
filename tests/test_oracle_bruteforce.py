"""Oracle pinned by brute force on tiny pools.

Schedule: every forced-action vector over n arrivals (actions -1..A-1) is run
through the oracle and through an independent list-based model
(tests/bruteforce.py); states must agree bit for bit over the following ticks.
Route: the oracle's masked argmax must equal an exhaustive fp64 enumeration of
all actions computed with numpy from the oracle's feature vector."""
import itertools

import numpy as np
import pytest

import oracle
import workload
from bruteforce import TinyPool
from helpers import tiny_cfg


def _arr(reqs):
    n = len(reqs)
    return dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32),
                budget=np.array([r[0] for r in reqs], np.int16),
                base_svc=np.array([r[1] for r in reqs], np.int16))


def _oracle(cfg, caps):
    A = cfg["A"]
    W = [np.zeros((w, i), np.float32) for w, i in zip(cfg["widths"], [cfg["feat_dim"]] + cfg["widths"][:-1])]
    b = [np.zeros(w, np.float32) for w in cfg["widths"]]
    emb = np.zeros((2, cfg["embed_dim"]), np.float32)
    return oracle.Oracle(cfg, W, b, emb, np.array([caps], np.int32))


def _compare(o, tp, ctx):
    s = o.state()
    bs = tp.snapshot()
    assert s["t"] == bs["t"], ctx
    for k in ("next_id", "arrived", "rej_nomodel"):
        assert int(s[k][0]) == bs[k], (ctx, k)
    for k in ("qlen", "busy", "ewma", "backlog", "rej_overflow", "enqueued", "started",
              "completed", "slo_met", "lat_sum", "wait_sum", "hist"):
        assert s[k][0].tolist() == bs[k], (ctx, k, s[k][0].tolist(), bs[k])
    for m in range(tp.M):
        assert s["queues"][0, m, :s["qlen"][0, m]].tolist() == bs["queues"][m], (ctx, m)
        assert s["slots"][0, m].tolist() == bs["slots"][m], (ctx, m)


@pytest.mark.parametrize("qcap,caps,mode", [(1, (1, 1), "slack"), (2, (1, 2), "slack"),
                                            (3, (2, 2), "slack"), (2, (2, 1), "deadline"),
                                            (3, (1, 2), "fcfs")])
def test_schedule_all_forced_actions(qcap, caps, mode):
    cfg = tiny_cfg(M=2, K=2, qcap=qcap, cap_hi=2, key_mode=mode)
    rng = np.random.default_rng(qcap * 10 + caps[0] + caps[1])
    history = []
    for _ in range(3):
        n = int(rng.integers(0, 4))
        history.append([(int(rng.integers(1, 12)), int(rng.integers(1, 4)),
                         int(rng.integers(-1, cfg["A"]))) for _ in range(n)])
    fields = [(int(rng.integers(1, 12)), int(rng.integers(1, 4))) for _ in range(4)]
    tail = [[(5, 1, 0)], [], []]
    for acts in itertools.product(range(-1, cfg["A"]), repeat=4):
        o = _oracle(cfg, caps)
        tp = TinyPool(2, 2, qcap, caps, mode, max_slots=cfg["max_slots"])
        ticks = history + [[(f[0], f[1], a) for f, a in zip(fields, acts)]] + tail
        for ti, reqs in enumerate(ticks):
            o.schedule(_arr([(r[0], r[1]) for r in reqs]), np.array([r[2] for r in reqs], np.int32))
            tp.step(reqs)
            if ti >= len(history):
                _compare(o, tp, (acts, ti))
        assert o.error == 0


def _relu(x):
    return np.maximum(x, 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_route_argmax_bruteforce(dtype):
    cfg = tiny_cfg(M=3, K=2, qcap=2, cap_hi=2, embed_dim=6, widths=[16, 6], dtype=dtype)
    rng = np.random.default_rng(7)
    W, b = workload.gen.weights(cfg, 3, 0.1)
    # rows 0..3 of the last layer duplicate row 0 -> exact logit ties
    W[1][1] = W[1][0]
    W[1][3] = W[1][0]
    b[1][1] = b[1][0]
    b[1][3] = b[1][0]
    emb = rng.standard_normal((8, 6)).astype(np.float32)
    if dtype == "bf16":
        emb = np.array([[oracle.round_bf16(v) for v in r] for r in emb], np.float32)
    o = oracle.Oracle(cfg, W, b, emb, np.array([[1, 2, 1]], np.int32))
    rb = oracle.round_bf16
    Wd = [np.vectorize(rb)(w.astype(np.float64)) if dtype == "bf16" else w.astype(np.float64) for w in W]
    for t in range(12):
        n = int(rng.integers(1, 5))
        arr = dict(offsets=np.array([0, n], np.int32), q_idx=rng.integers(0, 8, n).astype(np.int32),
                   budget=rng.integers(1, 20, n).astype(np.int16),
                   base_svc=rng.integers(1, 4, n).astype(np.int16))
        if t == 6:
            o.set_enabled(0, 2, 0)
        st = o.state()
        valid_m = [(st["qlen"][0, m] < cfg["qcap"]) and st["enabled"][0, m] and st["cap"][0, m] > 0
                   for m in range(cfg["M"])]
        act, lg = o.route(arr)
        for r in range(n):
            x = o.features(0, int(arr["q_idx"][r]), int(arr["budget"][r]))
            h = _relu(Wd[0] @ x + b[0].astype(np.float64))
            if dtype == "bf16":
                h = np.vectorize(rb)(h)
            z = Wd[1] @ h + b[1].astype(np.float64)
            np.testing.assert_allclose(lg[r], z, rtol=1e-12, atol=1e-12)
            best, bestv = -1, None
            for a in range(cfg["A"]):       # exhaustive, lowest index on ties
                if valid_m[a // cfg["K"]] and (bestv is None or z[a] > bestv):
                    best, bestv = a, z[a]
            assert act[r] == best, (t, r)
        o.schedule(arr, act)
    assert o.error == 0


def test_route_all_masked_rejects():
    cfg = tiny_cfg(M=2, K=2, qcap=1, cap_hi=1)
    W, b = workload.gen.weights(cfg, 0, 0.1)
    o = oracle.Oracle(cfg, W, b, np.zeros((2, cfg["embed_dim"]), np.float32), np.array([[1, 1]], np.int32))
    o.set_enabled(0, 0, 0)
    o.set_capacity(0, 1, 0)
    arr = _arr([(5, 1), (5, 1)])
    act, _ = o.route(arr)
    assert act.tolist() == [-1, -1]
    o.schedule(arr, act)
    s = o.state()
    assert s["rej_nomodel"][0] == 2 and s["arrived"][0] == 2 and s["qlen"].sum() == 0
