"""Oracle of the RL-rollout outputs pinned against published vectors, closed
forms and library routines.

* Philox4x32-10: the published known-answer vectors (tests/golden).
* Gumbel-max: the empirical distribution of sampled actions over many
  requests with identical logits matches the softmax of the logits over the
  valid actions (chi-square), and masked actions are never drawn.
* log pi and entropy: scipy's log-sum-exp / softmax over the valid actions;
  uniform logits give -ln(n_valid) and ln(n_valid).
* Greedy mode: the masked argmax of the plain route step.
* Value head: a torch fp64 linear chain with the value row appended; the
  policy logits do not change when the value row is added.
* Counters: env indices in the noise are global (an oracle over a slice of
  envs draws the same actions as one over all of them)."""
import json
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
import workload
from helpers import make_oracle, tiny_cfg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")


def test_philox_known_answers():
    with open(GOLDEN) as f:
        kat = json.load(f)
    for v in kat["vectors"]:
        ctr = [int(x, 16) for x in v["ctr"]]
        key = [int(x, 16) for x in v["key"]]
        out = [int(x, 16) for x in v["out"]]
        assert oracle.philox4x32_10(ctr, key).tolist() == out


def _same_request_tick(n, q=3, budget=50):
    return dict(offsets=np.array([0, n], np.int32), q_idx=np.full(n, q, np.int32),
                budget=np.full(n, budget, np.int16), base_svc=np.ones(n, np.int16))


def test_gumbel_max_samples_the_masked_softmax():
    n = 40000
    cfg = tiny_cfg(M=3, K=3, widths=[16, 9], max_arrivals=n, qcap=8)
    o, _ = make_oracle(cfg, seed=4, bias_scale=0.5, Q=8)
    o.set_enabled(0, 1, 0)                       # model 1 (actions 3..5) masked
    out = o.route_rl(_same_request_tick(n), seed=0x1234_5678_9ABC)
    z = out["logits"][0]
    assert np.all(out["logits"] == z)            # identical requests, identical logits
    valid = np.array([a // cfg["K"] != 1 for a in range(9)])
    p = np.zeros(9)
    p[valid] = scipy.special.softmax(z[valid])
    counts = np.bincount(out["actions"], minlength=9)
    assert counts[~valid].sum() == 0
    stat = ((counts[valid] - n * p[valid]) ** 2 / (n * p[valid])).sum()
    assert scipy.stats.chi2.sf(stat, valid.sum() - 1) > 1e-4, (counts, n * p)
    # every row's log-prob is that of its own action under the same softmax
    np.testing.assert_allclose(out["logp"], np.log(p[out["actions"]]), rtol=0, atol=1e-12)


def test_logp_entropy_match_scipy():
    cfg = workload.configs.get("c0", T=30)
    o, _ = make_oracle(cfg, seed=5, bias_scale=0.1, Q=64)
    cnt = workload.gen.counts(cfg, 5)
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 5, t, cnt[t], 64)
        if t % 7 == 3:
            o.set_enabled(0, t % cfg["M"], 0)
        out = o.route_rl(arr, seed=99 + t)
        s = o.state()
        valid = np.array([s["enabled"][0, a // cfg["K"]] != 0 and s["cap"][0, a // cfg["K"]] > 0
                          and s["qlen"][0, a // cfg["K"]] < cfg["qcap"] for a in range(cfg["A"])])
        for r in range(len(out["actions"])):
            z = out["logits"][r]
            if not valid.any():
                assert out["actions"][r] == -1 and out["logp"][r] == 0 and out["entropy"][r] == 0
                continue
            a = out["actions"][r]
            assert valid[a]
            lse = scipy.special.logsumexp(z[valid])
            assert abs(out["logp"][r] - (z[a] - lse)) < 1e-12
            pv = scipy.special.softmax(z[valid])
            assert abs(out["entropy"][r] - scipy.stats.entropy(pv)) < 1e-12
        o.schedule(arr, out["actions"])


def test_uniform_logits_closed_form():
    cfg = tiny_cfg(M=4, K=2, widths=[8, 8], max_arrivals=64)
    W, b = workload.gen.weights(cfg, 0, 0.0)
    W = [np.zeros_like(w) for w in W]             # every logit is 0
    _, emb = workload.gen.embedding(cfg, 0, rows=8)
    o = oracle.Oracle(cfg, W, b, emb, np.full((1, 4), 2, np.int32))
    o.set_enabled(0, 2, 0)
    out = o.route_rl(_same_request_tick(50), seed=7)
    nv = 6
    np.testing.assert_allclose(out["logp"], -np.log(nv), atol=1e-15)
    np.testing.assert_allclose(out["entropy"], np.log(nv), atol=1e-15)
    assert set(out["actions"].tolist()) <= {0, 1, 2, 3, 6, 7}


def test_greedy_mode_is_the_masked_argmax():
    cfg = workload.configs.get("c4", E=4, T=12)
    o, _ = make_oracle(cfg, seed=6, bias_scale=0.1, Q=64)
    cnt = workload.gen.counts(cfg, 6)
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 6, t, cnt[t], 64)
        act, lg = o.route(arr)
        out = o.route_rl(arr, seed=1, greedy=True)
        np.testing.assert_array_equal(out["actions"], act)
        np.testing.assert_array_equal(out["logits"], lg)
        o.schedule(arr, act)


def _torch_chain(cfg, W, b, x):
    F = torch.nn.functional
    h = torch.from_numpy(x)
    for l in range(len(W)):
        w = W[l].astype(np.float64)
        if cfg["dtype"] == "bf16":
            w = oracle.round_bf16_array(w).reshape(W[l].shape)
        h = F.linear(h, torch.from_numpy(w), torch.from_numpy(b[l].astype(np.float64)))
        if l + 1 < len(W):
            h = torch.relu(h)
            if cfg["dtype"] == "bf16":
                h = torch.from_numpy(oracle.round_bf16_array(h.numpy()))
    return h.numpy()


@pytest.mark.parametrize("name", ["c0", "c2", "c4"])
def test_value_head_matches_torch_linear(name):
    cfg = workload.configs.get(name, E=2, T=6, value_head=True)
    base = workload.configs.get(name, E=2, T=6)
    o, (W, b, emb, cap, lb) = make_oracle(cfg, seed=8, bias_scale=0.1, Q=64)
    o_plain, _ = make_oracle(base, seed=8, bias_scale=0.1, Q=64)
    A = cfg["A"]
    assert W[-1].shape[0] == A + 1
    cnt = workload.gen.counts(cfg, 8)
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 8, t, cnt[t], 64)
        out = o.route_rl(arr, seed=3)
        _, lg_plain = o_plain.route(arr)
        np.testing.assert_array_equal(out["logits"], lg_plain)
        for e in range(cfg["E"]):
            for r in range(arr["offsets"][e], arr["offsets"][e + 1]):
                x = o.features(e, int(arr["q_idx"][r]), int(arr["budget"][r]))
                y = _torch_chain(cfg, W, b, x)
                assert abs(out["value"][r] - y[A]) <= 1e-12 * max(1.0, abs(y[A]))
        o.schedule(arr, out["actions"])
        o_plain.schedule(arr, out["actions"])


def test_no_valid_action():
    cfg = tiny_cfg(M=2, K=2, value_head=True)
    o, _ = make_oracle(cfg, seed=9, Q=8)
    o.set_enabled(0, 0, 0)
    o.set_enabled(0, 1, 0)
    out = o.route_rl(_same_request_tick(5), seed=11)
    assert np.all(out["actions"] == -1) and np.all(out["logp"] == 0) and np.all(out["entropy"] == 0)
    assert np.all(out["value"] != 0)


def test_noise_uses_global_env_index():
    cfg = workload.configs.get("c2", E=6, T=4)
    o_all, (W, b, emb, cap, lb) = make_oracle(cfg, seed=10, Q=64)
    o_part = oracle.Oracle(cfg, W, b, emb, cap[3:5], lb, E=2)
    cnt = workload.gen.counts(cfg, 10)
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 10, t, cnt[t], 64)
        a_all = o_all.route_rl(arr, seed=2024)
        a_part = o_part.route_rl(workload.gen.subset(arr, 3, 5), seed=2024, env_base=3)
        lo, hi = arr["offsets"][3], arr["offsets"][5]
        np.testing.assert_array_equal(a_part["actions"], a_all["actions"][lo:hi])
        # a different seed changes the draws
        a_other = o_all.route_rl(arr, seed=2025)
        if t == 0:
            assert not np.array_equal(a_other["actions"], a_all["actions"])
        o_all.schedule(arr, a_all["actions"])
        o_part.schedule(workload.gen.subset(arr, 3, 5), a_part["actions"])
