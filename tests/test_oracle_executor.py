"""Pins of the oracle's dual-pathway executor (Sec. 4.2).

* The whole network against a chain of torch library layers in fp64
  (torch.nn.functional.linear / relu / layer_norm) fed with the oracle's own
  feature vector and role row, in fp32 and bf16 pools (<= 1e-12).
* LayerNorm in closed form: constant pre-activations with two levels give
  +-c with c = (u/2)/sqrt(u^2/4 + eps), which fixes the mean, the biased
  variance, the epsilon and that the ReLU comes before the normalisation.
* The budget head in closed form, and the system head's input order
  [queue depth | end-to-end latency | KV-cache use] against the state.
* Invariants: scaling the semantic (or resource) layer by 2 leaves the logits
  unchanged up to the epsilon; identical role rows give identical logits.
* Bad roles: action -1, error bit, the env untouched by the schedule step.
"""
import numpy as np
import pytest
import torch

import oracle
import workload
from helpers import make_oracle

F = torch.nn.functional
EPS = 1e-5


def _cfg(dtype="bf16", E=3, Ed=64, T=12, **kw):
    return workload.configs.get("c2d", E=E, T=T, embed_dim=Ed, dtype=dtype, **kw)


def _t(x):
    return torch.from_numpy(np.asarray(x, np.float64))


def _torch_executor(cfg, P, roles, x, role):
    """The executor of Sec. 4.2 as torch layers in fp64 on the feature vector x
    (query embedding, stat-major load statistics, budget)."""
    bf = cfg["dtype"] == "bf16"
    rnd = (lambda v: torch.from_numpy(oracle.round_bf16_array(v.numpy()))) if bf else (lambda v: v)
    W = {k: (rnd(_t(v)) if k.startswith("W_") else _t(v)) for k, v in P.items()}
    Ed, M = cfg["embed_dim"], cfg["M"]
    e_q = _t(x[:Ed])
    e_r = rnd(_t(roles[role]))
    h_sem = F.layer_norm(torch.relu(F.linear(torch.cat([e_q, e_r]), W["W_sem"], W["b_sem"])),
                         (128,), W["g_sem"], W["be_sem"], eps=EPS)
    h_sem = rnd(h_sem)
    b = _t(x[Ed + 4 * M:Ed + 4 * M + 1])
    h_bud = rnd(torch.relu(F.linear(b, W["W_bud"], W["b_bud"])))
    d_queue, d_kv, d_e2e = _t(x[Ed:Ed + M]), _t(x[Ed + M:Ed + 2 * M]), _t(x[Ed + 2 * M:Ed + 3 * M])
    h_sys = rnd(torch.relu(F.linear(torch.cat([d_queue, d_e2e, d_kv]), W["W_sys"], W["b_sys"])))
    h_res = F.layer_norm(torch.relu(F.linear(torch.cat([h_bud, h_sys]), W["W_res"], W["b_res"])),
                         (64,), W["g_res"], W["be_res"], eps=EPS)
    h_res = rnd(h_res)
    h = rnd(torch.relu(F.linear(torch.cat([h_sem, h_res]), W["W_merge"], W["b_merge"])))
    return F.linear(h, W["W_act"], W["b_act"]).numpy()


@pytest.mark.parametrize("dtype,Ed", [("f32", 64), ("bf16", 64), ("bf16", 384)])
def test_executor_matches_torch_layers(dtype, Ed):
    cfg = _cfg(dtype, Ed=Ed)
    o, (P, roles, emb, cap, lb) = make_oracle(cfg, seed=3, bias_scale=0.1, Q=64)
    cnt = workload.gen.counts(cfg, 3)
    A = cfg["A"]
    checked = 0
    for t in range(6):
        arr = workload.gen.tick(cfg, 3, t, cnt[t], 64)
        act, lg = o.route(arr)
        for e in range(cfg["E"]):
            for r in range(arr["offsets"][e], arr["offsets"][e + 1]):
                x = o.features(e, int(arr["q_idx"][r]), int(arr["budget"][r]))
                z = _torch_executor(cfg, P, roles, x, int(arr["role"][r]))
                np.testing.assert_allclose(lg[r], z[:A], rtol=1e-12, atol=1e-12)
                tr = o.dual_trace(e, int(arr["q_idx"][r]), int(arr["role"][r]), int(arr["budget"][r]))
                np.testing.assert_allclose(tr["z"], z, rtol=1e-12, atol=1e-12)
                checked += 1
        o.schedule(arr, act)
    assert checked > 50


def _const_params(cfg, **over):
    """Zero matrices, unit gains, zero biases; then the overrides."""
    Ed, M, A = cfg["embed_dim"], cfg["M"], cfg["A"]
    vh = 1 if cfg.get("value_head") else 0
    P = dict(W_sem=np.zeros((128, 2 * Ed)), b_sem=np.zeros(128), g_sem=np.ones(128), be_sem=np.zeros(128),
             W_bud=np.zeros((16, 1)), b_bud=np.zeros(16), W_sys=np.zeros((16, 3 * M)), b_sys=np.zeros(16),
             W_res=np.zeros((64, 32)), b_res=np.zeros(64), g_res=np.ones(64), be_res=np.zeros(64),
             W_merge=np.zeros((128, 192)), b_merge=np.zeros(128),
             W_act=np.zeros((A + vh, 128)), b_act=np.zeros(A + vh))
    P.update(over)
    return {k: np.asarray(v, np.float32) for k, v in P.items()}


def _oracle_with(cfg, P, seed=0):
    _, emb = workload.gen.embedding(cfg, seed, rows=32)
    cap = workload.gen.capacities(cfg, seed)
    return oracle.Oracle(cfg, P, None, emb, cap, None, roles=workload.gen.roles(cfg, seed))


def test_layer_norm_closed_form():
    """Two-level constant pre-activations: LN gives exactly +-(u/2)/sqrt(u^2/4 + eps)."""
    cfg = _cfg("f32")
    u = np.float32(0.01)
    gain = np.linspace(0.5, 1.5, 128).astype(np.float32)
    beta = np.linspace(-0.2, 0.2, 128).astype(np.float32)
    # rows 0..63 at u, rows 64..127 at -u: the ReLU maps the second half to 0
    b_sem = np.concatenate([np.full(64, u), np.full(64, -u)]).astype(np.float32)
    v = np.float32(0.25)
    b_res = np.concatenate([np.full(16, v), np.zeros(48)]).astype(np.float32)
    o = _oracle_with(cfg, _const_params(cfg, b_sem=b_sem, g_sem=gain, be_sem=beta, b_res=b_res))
    tr = o.dual_trace(0, 3, 1, 100)
    uu = float(u)
    c = (uu / 2) / np.sqrt(uu * uu / 4 + EPS)
    exp = np.concatenate([np.full(64, c), np.full(64, -c)]) * gain.astype(np.float64) + beta
    np.testing.assert_allclose(tr["h_sem"], exp, rtol=1e-13, atol=1e-15)
    # resource pathway: 16 of 64 at v, mean v/4, biased variance 3 v^2 / 16
    vv = float(v)
    mean, var = vv / 4, 3 * vv * vv / 16
    exp_r = np.concatenate([np.full(16, (vv - mean)), np.full(48, -mean)]) / np.sqrt(var + EPS)
    np.testing.assert_allclose(tr["h_res"], exp_r, rtol=1e-13, atol=1e-15)
    # all-zero input to a LayerNorm: the output is its bias
    o2 = _oracle_with(cfg, _const_params(cfg, be_sem=beta))
    np.testing.assert_allclose(o2.dual_trace(0, 3, 1, 100)["h_sem"], beta.astype(np.float64), rtol=0, atol=0)


def test_budget_and_system_heads_closed_form():
    cfg = _cfg("f32", E=2, T=40)
    M, B = cfg["M"], cfg["budget_max"]
    W_bud = np.linspace(-1, 1, 16).astype(np.float32).reshape(16, 1)
    b_bud = np.linspace(0.3, -0.3, 16).astype(np.float32)
    # system head: row 3 m + s reads input m + M s (the paper's order queue | e2e | kv)
    W_sys = np.zeros((16, 3 * M), np.float32)
    for m in range(M):
        for s in range(3):
            W_sys[3 * m + s, s * M + m] = 1.0
    P = _const_params(cfg, W_bud=W_bud, b_bud=b_bud, W_sys=W_sys)
    o = _oracle_with(cfg, P, seed=4)
    cnt = workload.gen.counts(cfg, 4)
    for t in range(40):
        # the policy is constant: enable one model per tick so every model gets load
        for e in range(cfg["E"]):
            for m in range(M):
                o.set_enabled(e, m, m == t % M)
        o.tick(workload.gen.tick(cfg, 4, t, cnt[t], 32))
    s = o.state()
    f32 = np.float32
    for budget in (1, 77, 400):
        tr = o.dual_trace(1, 5, 0, budget)
        bfeat = float(f32(budget) * f32(1.0 / B))
        exp = np.maximum(W_bud[:, 0].astype(np.float64) * bfeat + b_bud, 0.0)
        np.testing.assert_allclose(tr["h_bud"], exp, rtol=1e-15, atol=0)
    tr = o.dual_trace(1, 5, 0, 50)
    assert np.all(s["qlen"][1] > 0) and np.all(s["busy"][1] > 0) and np.all(s["ewma"][1] > 0)
    for m in range(M):
        c = max(int(s["cap"][1, m]), 1)
        q = float(f32(s["qlen"][1, m]) * f32(1.0 / cfg["qcap"]))
        lat = float(f32(s["ewma"][1, m]) * f32(1.0 / (256.0 * B)))
        kv = float(f32(s["busy"][1, m]) * f32(1.0 / c))
        assert tr["h_sys"][3 * m + 0] == q, m
        assert tr["h_sys"][3 * m + 1] == lat, m
        assert tr["h_sys"][3 * m + 2] == kv, m


@pytest.mark.parametrize("which", ["sem", "res"])
def test_layer_norm_scale_invariance(which):
    """Doubling a LayerNorm'd layer's weights and bias changes only the
    epsilon's share of the normaliser."""
    cfg = _cfg("f32", E=2)
    P = workload.gen.dual_weights(cfg, 6, 0.1)
    roles = workload.gen.roles(cfg, 6)
    _, emb = workload.gen.embedding(cfg, 6, rows=32)
    cap = workload.gen.capacities(cfg, 6)
    P2 = dict(P)
    P2[f"W_{which}"] = P[f"W_{which}"] * 2
    P2[f"b_{which}"] = P[f"b_{which}"] * 2
    o1 = oracle.Oracle(cfg, P, None, emb, cap, roles=roles)
    o2 = oracle.Oracle(cfg, P2, None, emb, cap, roles=roles)
    cnt = workload.gen.counts(cfg, 6)
    for t in range(5):
        arr = workload.gen.tick(cfg, 6, t, cnt[t], 32)
        a1, l1 = o1.route(arr)
        a2, l2 = o2.route(arr)
        np.testing.assert_allclose(l1, l2, rtol=0, atol=2e-3 * np.abs(l1).max())
        o1.schedule(arr, a1)
        o2.schedule(arr, a1)


def test_role_enters_only_through_its_embedding():
    cfg = _cfg("bf16", E=2)
    P = workload.gen.dual_weights(cfg, 7, 0.1)
    roles = workload.gen.roles(cfg, 7)
    roles[5] = roles[2]
    _, emb = workload.gen.embedding(cfg, 7, rows=32)
    o = oracle.Oracle(cfg, P, None, emb, workload.gen.capacities(cfg, 7), roles=roles)
    z2 = o.dual_trace(0, 4, 2, 90)["z"]
    np.testing.assert_array_equal(z2, o.dual_trace(0, 4, 5, 90)["z"])
    assert not np.array_equal(z2, o.dual_trace(0, 4, 3, 90)["z"])
    # the query embedding matters too
    assert not np.array_equal(z2, o.dual_trace(0, 9, 2, 90)["z"])


def test_bad_role_rejected_env_untouched():
    cfg = _cfg("bf16", E=3)
    o, _ = make_oracle(cfg, seed=8, Q=32)
    cnt = workload.gen.counts(cfg, 8)
    for t in range(3):
        o.tick(workload.gen.tick(cfg, 8, t, cnt[t], 32))
    arr = workload.gen.tick(cfg, 8, 3, np.array([3, 2, 4], np.int32), 32)
    arr["role"] = arr["role"].copy()
    arr["role"][3] = cfg["n_roles"]           # env 1's first row
    before = o.state()
    act, lg = o.route(arr)
    assert act[3] == -1 and np.all(lg[3] == 0)
    assert o.error & oracle.ERR_ROLE
    o.schedule(arr, act)
    after = o.state()
    for k in ("qlen", "busy", "enqueued", "next_id"):
        if k in before:
            np.testing.assert_array_equal(np.asarray(after[k])[1], np.asarray(before[k])[1], err_msg=k)
    assert after["next_id"][0] != before["next_id"][0]
    arr["role"][3] = -1
    o.clear_error()
    o.route(arr)
    assert o.error & oracle.ERR_ROLE
