"""Shared test helpers: pool construction from a workload config, state
comparison, and the logit tolerance rule of the tick's parity contract."""
from __future__ import annotations

import numpy as np

import oracle
import workload

STATE_INT_KEYS = ("next_id", "arrived", "rej_nomodel", "qlen", "busy", "ewma", "backlog", "cost_q16",
                  "rpm_limit", "rpm_count", "rpm_hist",
                  "cap", "enabled", "rej_overflow", "enqueued", "started", "completed",
                  "slo_met", "lat_sum", "wait_sum", "hist", "slots")


def tiny_cfg(M=2, K=2, qcap=3, cap_hi=2, embed_dim=4, widths=None, dtype="f32",
             key_mode="slack", budget_hi=20, E=1, max_arrivals=64, **kw):
    A = M * K
    widths = widths or [8, A]
    cfg = dict(index=0, E=E, M=M, K=K, qcap=qcap, cap_lo=1, cap_hi=cap_hi, budget_lo=1,
               budget_hi=budget_hi, embed_dim=embed_dim,
               feat_dim=embed_dim + 4 * M + 1, widths=widths, dtype=dtype, key_mode=key_mode,
               max_arrivals=max_arrivals, lam=2.0, T=10, svc_mu=0.5, svc_sigma=0.5, zipf_s=None)
    cfg.update(kw)
    return workload.configs.finish(cfg)


def make_oracle(cfg, seed=0, bias_scale=0.1, Q=None, E=None, cap=None, threads=1):
    """Oracle pool of cfg with seeded inputs. For the dual-pathway executor W
    is the parameter dict and b the role-embedding table."""
    if cfg.get("net") == "dual":
        W, b = workload.gen.dual_weights(cfg, seed, bias_scale), workload.gen.roles(cfg, seed)
    else:
        W, b = workload.gen.weights(cfg, seed, bias_scale)
    _, emb = workload.gen.embedding(cfg, seed, rows=Q)
    cap = workload.gen.capacities(cfg, seed) if cap is None else cap
    lb = workload.gen.logit_bias(cfg)
    o = oracle.Oracle(cfg, W, b, emb, cap, lb, E=E, threads=threads,
                      roles=b if cfg.get("net") == "dual" else None)
    return o, (W, b, emb, cap, lb)


def assert_state_equal(a: dict, b: dict, envs=None, ctx=""):
    """Bit-exact comparison of two state snapshots (same layout)."""
    assert a["t"] == b["t"], ctx
    sel = slice(None) if envs is None else envs
    for k in STATE_INT_KEYS:
        x, y = np.asarray(a[k])[sel], np.asarray(b[k])[sel]
        if not np.array_equal(x, y):
            idx = np.argwhere(x != y)[:5]
            raise AssertionError(f"{ctx}: state field {k} differs at {idx.tolist()}: "
                                 f"{x[tuple(idx[0])]} vs {y[tuple(idx[0])]}")
    qa, qb = np.asarray(a["queues"])[sel], np.asarray(b["queues"])[sel]
    ql = np.asarray(a["qlen"])[sel]
    E, M = ql.shape
    for e in range(E):
        for m in range(M):
            n = int(ql[e, m])
            if not np.array_equal(qa[e, m, :n], qb[e, m, :n]):
                d = np.argwhere(np.any(qa[e, m, :n] != qb[e, m, :n], axis=-1))[:3]
                raise AssertionError(f"{ctx}: queue (env {e}, model {m}) differs at "
                                     f"positions {d.ravel().tolist()}")


def logits_close(g: np.ndarray, o: np.ndarray, rtol: float):
    """Row-wise rule: |g_a - o_a| <= rtol * max_b |o_b| for every a.
    Returns a boolean mask of passing rows."""
    scale = np.max(np.abs(o), axis=1, keepdims=True)
    return np.all(np.abs(g - o) <= rtol * scale + 1e-30, axis=1)


def near_tie(o_row: np.ndarray, a_oracle: int, a_gpu: int, rtol: float) -> bool:
    """Two argmaxes may differ only if the oracle's margin between them is
    within twice the logit tolerance."""
    if a_oracle < 0 or a_gpu < 0:
        return False
    scale = np.max(np.abs(o_row))
    return o_row[a_oracle] - o_row[a_gpu] <= 2 * rtol * scale


def check_invariants(s: dict, cfg: dict, prev: dict | None = None, ctx=""):
    """Closed-form invariants of the tick on a state snapshot (every env).

    Conservation of requests, sorted queues, capacity bounds, backlog as the
    sum of queued service times, key formula per mode and id uniqueness.
    With `prev` (the snapshot one tick earlier) also work conservation: a slot
    below c_m may be empty while the queue is non-empty only if it completed
    a request this tick."""
    E, M = s["qlen"].shape
    K, qcap = cfg["K"], cfg["qcap"]
    mode = cfg["key_mode"]
    fail = lambda msg: AssertionError(f"{ctx}: {msg}")  # noqa: E731
    tot_rej = s["rej_overflow"].sum(1)
    tot_enq = s["enqueued"].sum(1)
    if not np.array_equal(s["arrived"], s["rej_nomodel"] + tot_rej + tot_enq):
        raise fail("arrived != rejected + enqueued")
    if not np.array_equal(s["enqueued"], s["qlen"] + s["started"]):
        raise fail("enqueued != qlen + started")
    if not np.array_equal(s["started"], s["busy"] + s["completed"]):
        raise fail("started != busy + completed")
    if not np.array_equal(s["hist"].sum(1), s["arrived"] - s["rej_nomodel"]):
        raise fail("histogram total != routed requests")
    if np.any(s["qlen"] > qcap) or np.any(s["qlen"] < 0):
        raise fail("qlen out of [0, QCAP]")
    if np.any(s["slo_met"] > s["completed"]) or np.any(s["ewma"] < 0):
        raise fail("slo_met > completed or negative EWMA")
    for e in range(E):
        for m in range(M):
            n = int(s["qlen"][e, m])
            q = s["queues"][e, m, :n].astype(np.int64)
            if n > 1:
                kk = q[:, 0] * (1 << 32) + q[:, 1]
                if not np.all(np.diff(kk) > 0):
                    raise fail(f"queue ({e},{m}) not strictly increasing in (key, id)")
            if int(q[:, 3].sum()) != int(s["backlog"][e, m]):
                raise fail(f"backlog ({e},{m}) != sum of queued svc")
            if n:
                if mode == "slack":
                    exp = q[:, 2] + q[:, 4] - q[:, 3]
                elif mode == "deadline":
                    exp = q[:, 2] + q[:, 4]
                else:
                    exp = q[:, 2]
                if not np.array_equal(q[:, 0], exp):
                    raise fail(f"queue ({e},{m}) key formula")
                if np.any(q[:, 1] >= s["next_id"][e]) or np.any(q[:, 2] >= s["t"]):
                    raise fail(f"queue ({e},{m}) id/t_arr from the future")
            sl = s["slots"][e, m]
            busy = int(np.sum(sl[:, 0] >= 0))
            if busy != int(s["busy"][e, m]):
                raise fail(f"busy count ({e},{m})")
            if np.any(sl[sl[:, 0] >= 0, 2] < 1):
                raise fail(f"busy slot with rem < 1 ({e},{m})")
            c = int(s["cap"][e, m])
            held = "rpm_limit" in s and 0 < int(s["rpm_limit"][e, m]) <= int(s["rpm_count"][e, m])
            if prev is not None and n > 0 and int(prev["cap"][e, m]) == c and not held:
                empty = int(np.sum(sl[:c, 0] < 0))
                done = int(s["completed"][e, m] - prev["completed"][e, m])
                if empty > done:
                    raise fail(f"idle slot with non-empty queue ({e},{m})")
        ids = np.concatenate([s["queues"][e, m, :s["qlen"][e, m], 1] for m in range(M)] +
                             [s["slots"][e, m][s["slots"][e, m][:, 0] >= 0, 0] for m in range(M)])
        if len(np.unique(ids)) != len(ids):
            raise fail(f"duplicate request id in env {e}")
