"""The five benchmark pools of the route-and-schedule tick, with every reading
the paper leaves open written down as a field.

Units (Sec. 5.1 evaluation protocol, restated for a discrete simulator): one
tick stands for one scheduling interval; arrivals per env are Poisson(lam) per
tick; budgets and service times are integer ticks.

Fields
------
E          independent simulated serving pools ("envs")
M, K       models and reasoning-depth levels; A = M*K joint actions
           (Sec. 3 "Action": a decodes to model a // K and depth a % K)
lam, T     Poisson arrivals per env-tick, ticks per run
qcap       per-(env, model) queue capacity
cap_lo/hi  service slots c_m drawn uniformly in [cap_lo, cap_hi]; max_slots = cap_hi
           (Table 5: vLLM serves up to max_num_seqs sequences at once; here c_m
           concurrent slots, an M/G/c station)
budget_lo/hi   request budget drawn uniformly in [lo, hi] ticks (Sec. 3 "State":
           beta, the time budget); budget_max = budget_hi normalises features
svc_mu/sigma   base service time ceil(lognormal(mu, sigma)), clamped to SVC_MAX;
           a request served at depth d takes base_svc*(d+1) ticks
embed_dim  query-embedding width E_d (Sec. 3: Sentence-BERT vectors; here N(0,1))
feat_dim   policy input width D_in; the features are
           [embedding | 4 load stats per model | remaining budget | zero pad]
widths     layer output widths of the policy MLP, last = A
net        "mlp" (default) or "dual": the paper's dual-pathway executor (Sec. 4.2),
           whose widths are the paper's (128 / 16 / 16 / 64 / 128); it reads the
           query embedding, a role embedding (n_roles rows, one role per
           request), the remaining budget and three of the load statistics
n_roles    rows of the role-embedding table (dual-pathway executor)
max_steps  > 1: multi-step agent chains (Sec. 4.3): each query is a sequence of
           n_steps calls, n_steps uniform in [1, max_steps]; the completion of a
           call spawns the next, routed at the following tick with what is left
           of the query's budget (the query's deadline is inherited)
value_head when true, the policy has a value row V(s) besides the A logits
q_rows_cap upper bound on the embedding-table rows (default 2^22)
dtype      "f32" or "bf16" (bf16 weights/activations, fp32 accumulate)
zipf_s     when set, a per-model logit bias -s*ln(m+1) (unnormalised Zipf log-pmf)
key_mode   "slack" (latest start time), "deadline" (EDF, Sec. 4.3) or "fcfs"
"""
from __future__ import annotations

import copy

SVC_MAX = 1023          # clamp of the base service time (ticks)
BUDGET_MAX_FIELD = 32767  # budgets travel as int16
Q_CAP_ROWS = 1 << 22    # embedding-table rows are min(total requests, 2^22)

_BASE = dict(
    M=5, K=3, key_mode="slack", zipf_s=None,
    cap_lo=1, cap_hi=3, budget_lo=20, budget_hi=400,
    svc_mu=1.0, svc_sigma=0.5, max_arrivals=1024,
)

CONFIGS = {
    # 1 env, correctness and launch-latency case
    "c0": dict(_BASE, index=0, E=1, lam=4.0, T=100, qcap=256,
               budget_hi=200, embed_dim=32, feat_dim=54, widths=[64, 15],
               dtype="f32"),
    # 1024 envs, fp32 policy
    "c1": dict(_BASE, index=1, E=1024, lam=16.0, T=200, qcap=1024,
               embed_dim=64, feat_dim=86, widths=[256, 256, 15], dtype="f32"),
    # 4096 envs, bf16 policy, load sweep lam in {4, 16, 64}
    "c2": dict(_BASE, index=2, E=4096, lam=64.0, T=256, qcap=2048,
               embed_dim=64, feat_dim=86, widths=[256, 256, 15], dtype="bf16",
               lam_sweep=[4.0, 16.0, 64.0]),
    # 4096 envs, 16 models x 4 depths, wide policy, heavy-tailed service
    "c3": dict(_BASE, index=3, E=4096, M=16, K=4, lam=64.0, T=256, qcap=4096,
               svc_mu=1.5, svc_sigma=1.0, embed_dim=128, feat_dim=193,
               widths=[512, 512, 64], dtype="bf16"),
    # 65536 envs, overload with overflow rejections and a Zipf model bias
    "c4": dict(_BASE, index=4, E=65536, M=8, K=3, lam=128.0, T=128, qcap=512,
               cap_lo=1, cap_hi=2, embed_dim=64, feat_dim=104,
               widths=[256, 24], dtype="bf16", zipf_s=1.2),
    # c2's pools with the paper's dual-pathway executor (Sec. 4.2): 384-d query
    # and role embeddings (Sentence-BERT width), 8 roles, 5 models x 3
    # strategies, a value head; 2^20 table rows (768 MB in bf16)
    # c2's pools running multi-step agent chains: 16 queries per env-tick of
    # 1-4 sequential calls (about 40 calls per env-tick), deadlines inherited
    "c2c": dict(_BASE, index=6, E=4096, lam=16.0, T=256, qcap=2048, max_steps=4,
                embed_dim=64, feat_dim=86, widths=[256, 256, 15], dtype="bf16"),
    "c2d": dict(_BASE, index=5, E=4096, lam=64.0, T=256, qcap=2048, net="dual",
                embed_dim=384, n_roles=8, value_head=True, dtype="bf16",
                q_rows_cap=1 << 20, lam_sweep=[4.0, 16.0, 64.0]),
}


def get(name: str, **overrides) -> dict:
    """A deep copy of config `name` with `overrides` applied and derived
    fields (A, max_slots, budget_max, n_layers) filled in."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg["name"] = name
    return finish(cfg)


def finish(cfg: dict) -> dict:
    cfg["A"] = cfg["M"] * cfg["K"]
    cfg["max_slots"] = cfg["cap_hi"]
    cfg["budget_max"] = cfg["budget_hi"]
    if cfg.get("net", "mlp") == "dual":
        # the executor reads [emb | 4 load stats per model | budget] like the MLP
        cfg["feat_dim"] = cfg["embed_dim"] + 4 * cfg["M"] + 1
        cfg["widths"] = None
        cfg["n_layers"] = None
        return cfg
    cfg["net"] = "mlp"
    cfg["n_layers"] = len(cfg["widths"])
    if cfg["widths"][-1] != cfg["A"]:
        raise ValueError("last layer width must equal M*K")
    if cfg["feat_dim"] < cfg["embed_dim"] + 4 * cfg["M"] + 1:
        raise ValueError("feat_dim too small for [emb | 4M stats | budget]")
    return cfg


def small(name: str, E: int | None = None, T: int | None = None, **kw) -> dict:
    """A reduced copy for tests: fewer envs/ticks, same shapes otherwise."""
    over = dict(kw)
    if E is not None:
        over["E"] = E
    if T is not None:
        over["T"] = T
    return get(name, **over)
