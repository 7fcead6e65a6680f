"""Seeded synthetic inputs for the route-and-schedule tick.

This module only draws random inputs: policy weights, service capacities, the
query-embedding table, Poisson arrival counts and per-request fields. It holds
none of the tick's arithmetic (no features, no policy evaluation, no keys, no
queue logic), so the oracle and the GPU path can both consume it without
sharing any part of the method.

Streams: numpy.random.default_rng(SeedSequence([seed, cfg index, stream]))
  0 weights, 1 capacities, 2 embedding table, 3 Poisson counts [T, E],
  4 request fields, one sub-stream per tick: SeedSequence([seed, idx, 4, t]),
  5 the value-head row (pools with cfg["value_head"]),
  6 the dual-pathway executor's parameters, 7 its role-embedding table,
  8 per-tick role of each request: SeedSequence([seed, idx, 8, t]),
  9 per-tick number of calls of each query (chain pools): SeedSequence([seed, idx, 9, t]).

Inputs stand in for the paper's workloads (Sec. 5.1): the paper's LLM-quality
benchmarks are replaced by N(0,1) query embeddings (Sec. 3 uses Sentence-BERT
vectors), its req/min Poisson rates by per-env Poisson(lam) per tick.
"""
from __future__ import annotations

import math

import numpy as np

from . import configs as _configs


def _rng(cfg: dict, seed: int, *stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg["index"], *stream]))


def table_rows(cfg: dict) -> int:
    """Embedding-table rows: min(expected total requests, 2^22), at least 16."""
    total = int(math.ceil(cfg["lam"] * cfg["E"] * cfg["T"]))
    return max(16, min(total, cfg.get("q_rows_cap", _configs.Q_CAP_ROWS)))


def weights(cfg: dict, seed: int = 0, bias_scale: float = 0.0):
    """Glorot-uniform fp32 weights [out, in] per layer and fp32 biases.

    Biases are U(-bias_scale, bias_scale) (0 in benchmarks, 0.1 in tests).
    With cfg["value_head"], one more row (the value head, its own stream,
    Glorot-uniform with fan_out 1) is appended to the last layer, so the
    policy rows are the same with and without it."""
    rng = _rng(cfg, seed, 0)
    Ws, bs = [], []
    fan_in = cfg["feat_dim"]
    for out in cfg["widths"]:
        lim = math.sqrt(6.0 / (fan_in + out))
        Ws.append(rng.uniform(-lim, lim, size=(out, fan_in)).astype(np.float32))
        if bias_scale > 0:
            bs.append(rng.uniform(-bias_scale, bias_scale, size=out).astype(np.float32))
        else:
            bs.append(np.zeros(out, np.float32))
        fan_in = out
    if cfg.get("value_head"):
        vr = _rng(cfg, seed, 5)
        h_last = Ws[-1].shape[1]
        lim = math.sqrt(6.0 / (h_last + 1))
        w_val = vr.uniform(-lim, lim, size=(1, h_last)).astype(np.float32)
        b_val = (vr.uniform(-bias_scale, bias_scale, size=1) if bias_scale > 0
                 else np.zeros(1)).astype(np.float32)
        Ws[-1] = np.concatenate([Ws[-1], w_val], axis=0)
        bs[-1] = np.concatenate([bs[-1], b_val])
    return Ws, bs


def _glorot(rng, out, fan_in):
    lim = math.sqrt(6.0 / (fan_in + out))
    return rng.uniform(-lim, lim, size=(out, fan_in)).astype(np.float32)


def dual_weights(cfg: dict, seed: int = 0, bias_scale: float = 0.0) -> dict:
    """Parameters of the dual-pathway executor (Sec. 4.2) as fp32 arrays:
    Glorot-uniform matrices [out, in], biases U(-bias_scale, bias_scale) (0 when
    bias_scale is 0), LayerNorm gains 1 + U(-bias_scale, bias_scale) and
    LayerNorm biases U(-bias_scale, bias_scale). Widths: W_sem 128 x 2E_d,
    W_bud 16 x 1, W_sys 16 x 3M, W_res 64 x 32, W_merge 128 x 192, W_act
    A x 128; with cfg["value_head"] one more W_act row (the value head, drawn
    from its own stream)."""
    rng = _rng(cfg, seed, 6)
    Ed, M, A = cfg["embed_dim"], cfg["M"], cfg["A"]

    def vec(n, center=0.0):
        if bias_scale > 0:
            return (center + rng.uniform(-bias_scale, bias_scale, size=n)).astype(np.float32)
        return np.full(n, center, np.float32)

    p = {}
    p["W_sem"] = _glorot(rng, 128, 2 * Ed); p["b_sem"] = vec(128)
    p["g_sem"] = vec(128, 1.0); p["be_sem"] = vec(128)
    p["W_bud"] = _glorot(rng, 16, 1); p["b_bud"] = vec(16)
    p["W_sys"] = _glorot(rng, 16, 3 * M); p["b_sys"] = vec(16)
    p["W_res"] = _glorot(rng, 64, 32); p["b_res"] = vec(64)
    p["g_res"] = vec(64, 1.0); p["be_res"] = vec(64)
    p["W_merge"] = _glorot(rng, 128, 192); p["b_merge"] = vec(128)
    p["W_act"] = _glorot(rng, A, 128); p["b_act"] = vec(A)
    if cfg.get("value_head"):
        vr = _rng(cfg, seed, 5)
        lim = math.sqrt(6.0 / (128 + 1))
        w_val = vr.uniform(-lim, lim, size=(1, 128)).astype(np.float32)
        b_val = (vr.uniform(-bias_scale, bias_scale, size=1) if bias_scale > 0
                 else np.zeros(1)).astype(np.float32)
        p["W_act"] = np.concatenate([p["W_act"], w_val], axis=0)
        p["b_act"] = np.concatenate([p["b_act"], b_val])
    return p


def roles(cfg: dict, seed: int = 0) -> np.ndarray:
    """Role-embedding table [n_roles, E_d] of N(0,1) fp32 values (Sec. 4.2 uses
    Sentence-BERT vectors of the role descriptions)."""
    rng = _rng(cfg, seed, 7)
    return rng.standard_normal(size=(cfg["n_roles"], cfg["embed_dim"]), dtype=np.float32)


def capacities(cfg: dict, seed: int = 0) -> np.ndarray:
    """Service slots c_m per (env, model): int32 [E, M], uniform in [cap_lo, cap_hi]."""
    rng = _rng(cfg, seed, 1)
    return rng.integers(cfg["cap_lo"], cfg["cap_hi"] + 1,
                        size=(cfg["E"], cfg["M"])).astype(np.int32)


def embedding(cfg: dict, seed: int = 0, rows: int | None = None):
    """Query-embedding table [Q, E_d] of N(0,1) values.

    Returns (table, values): for fp32 configs both are the same float32 array;
    for bf16 configs `table` holds the bf16 bit patterns (uint16, rounded to
    nearest-even by torch's conversion) and `values` the float32 value of each."""
    Q = table_rows(cfg) if rows is None else rows
    rng = _rng(cfg, seed, 2)
    x = rng.standard_normal(size=(Q, cfg["embed_dim"]), dtype=np.float32)
    if cfg["dtype"] == "f32":
        return x, x
    import torch
    t = torch.from_numpy(x).to(torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16).copy()
    vals = t.to(torch.float32).numpy()
    return bits, vals


def counts(cfg: dict, seed: int = 0) -> np.ndarray:
    """Poisson(lam) arrivals per (tick, env): int32 [T, E]."""
    rng = _rng(cfg, seed, 3)
    c = rng.poisson(cfg["lam"], size=(cfg["T"], cfg["E"]))
    return np.minimum(c, cfg["max_arrivals"]).astype(np.int32)


def tick(cfg: dict, seed: int, t: int, counts_row: np.ndarray, Q: int):
    """Arrival records of tick t for all envs, in env-major (CSR) order.

    Returns dict(offsets int32 [E+1], q_idx int32 [n], budget int16 [n],
    base_svc int16 [n]). Within an env, records are in arrival order."""
    rng = _rng(cfg, seed, 4, t)
    n = int(counts_row.sum())
    offsets = np.zeros(len(counts_row) + 1, np.int32)
    np.cumsum(counts_row, out=offsets[1:])
    q_idx = rng.integers(0, Q, size=n).astype(np.int32)
    budget = rng.integers(cfg["budget_lo"], cfg["budget_hi"] + 1, size=n).astype(np.int16)
    ln = rng.lognormal(cfg["svc_mu"], cfg["svc_sigma"], size=n)
    base_svc = np.minimum(np.ceil(ln), _configs.SVC_MAX).astype(np.int16)
    base_svc = np.maximum(base_svc, 1).astype(np.int16)
    out = dict(offsets=offsets, q_idx=q_idx, budget=budget, base_svc=base_svc)
    if cfg.get("n_roles"):
        rr = _rng(cfg, seed, 8, t)
        out["role"] = rr.integers(0, cfg["n_roles"], size=n).astype(np.int16)
    if cfg.get("max_steps", 1) > 1:
        rs = _rng(cfg, seed, 9, t)
        out["n_steps"] = rs.integers(1, cfg["max_steps"] + 1, size=n).astype(np.int16)
    return out


def subset(arr: dict, e0: int, e1: int) -> dict:
    """The records of envs [e0, e1) of one tick, offsets rebased to 0."""
    off = arr["offsets"]
    lo, hi = int(off[e0]), int(off[e1])
    out = dict(offsets=(off[e0:e1 + 1] - lo).astype(np.int32),
               q_idx=arr["q_idx"][lo:hi], budget=arr["budget"][lo:hi],
               base_svc=arr["base_svc"][lo:hi])
    for k in ("role", "n_steps"):
        if k in arr:
            out[k] = arr[k][lo:hi]
    return out


def logit_bias(cfg: dict):
    """Per-model logit bias -s*ln(m+1) as float32 [M], or None."""
    s = cfg.get("zipf_s")
    if not s:
        return None
    return np.array([-s * math.log(m + 1) for m in range(cfg["M"])], np.float32)


def trace(cfg: dict, seed: int = 0, Q: int | None = None, T: int | None = None):
    """All ticks of a run: list of per-tick dicts (small configs only)."""
    Q = table_rows(cfg) if Q is None else Q
    cnt = counts(cfg, seed)
    T = cfg["T"] if T is None else T
    return [tick(cfg, seed, t, cnt[t], Q) for t in range(T)]
