"""Oracle numerics pinned to library routines.

* bf16 rounding: the oracle's round-to-nearest-even must equal torch's
  fp32 -> bfloat16 conversion on random bit patterns and on the edge cases
  (ties, subnormals, largest finite, overflow).
* Policy MLP: the oracle's fp64 logits must equal a torch.nn.functional.linear
  chain in fp64 fed with the oracle's own feature vector (<= 1e-12)."""
import numpy as np
import pytest
import torch

import oracle
import workload
from helpers import make_oracle


def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_random_bit_patterns():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2**32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    np.testing.assert_array_equal(oracle.round_bf16_array(x.astype(np.float64)), _torch_bf16(x))


def test_bf16_edge_cases():
    f = np.float32
    cases = [1.0 + 2.0**-8, 1.0 + 3 * 2.0**-8, -(1.0 + 2.0**-8), 1.0 + 2.0**-8 + 2.0**-20,
             2.0**-126, 2.0**-130, 2.0**-133, 3 * 2.0**-134, 2.0**-149, -2.0**-140,
             float(np.finfo(np.float32).max), 3.3895313892515355e38, 3.39e38, 0.0, -0.0,
             0.1, 0.2, 0.3, 1e-3, 65504.0, 1.0 / 3.0]
    x = np.array(cases, f)
    np.testing.assert_array_equal(oracle.round_bf16_array(x.astype(np.float64)), _torch_bf16(x))
    # every exponent, mantissa patterns around the rounding point
    m = np.array([0x7FFF, 0x8000, 0x8001, 0x17FFF, 0x18000, 0x18001], np.uint32)
    e = np.arange(0, 255, dtype=np.uint32)
    b = ((e[:, None] << 23) | m[None, :]).ravel()
    x = np.concatenate([b, b | 0x80000000]).view(np.float32)
    x = x[np.isfinite(x)]
    np.testing.assert_array_equal(oracle.round_bf16_array(x.astype(np.float64)), _torch_bf16(x))


def _torch_mlp(o, cfg, W, b, x, lb):
    F = torch.nn.functional
    h = torch.from_numpy(x)
    L = len(W)
    for l in range(L):
        w = torch.from_numpy(W[l].astype(np.float64))
        if cfg["dtype"] == "bf16":
            w = torch.from_numpy(oracle.round_bf16_array(W[l].astype(np.float64)).reshape(W[l].shape))
        h = F.linear(h, w, torch.from_numpy(b[l].astype(np.float64)))
        if l + 1 < L:
            h = torch.relu(h)
            if cfg["dtype"] == "bf16":
                h = torch.from_numpy(oracle.round_bf16_array(h.numpy()))
    z = h.numpy()
    if lb is not None:
        z = z + np.repeat(lb.astype(np.float64), cfg["K"])
    return z


@pytest.mark.parametrize("name", ["c0", "c1", "c2", "c3", "c4"])
def test_mlp_matches_torch_linear(name):
    cfg = workload.configs.get(name, E=2, T=8)
    o, (W, b, emb, cap, lb) = make_oracle(cfg, seed=1, bias_scale=0.1, Q=64)
    cnt = workload.gen.counts(cfg, 1)
    for t in range(3):
        arr = workload.gen.tick(cfg, 1, t, cnt[t], 64)
        act, lg = o.route(arr)
        for e in range(cfg["E"]):
            for r in range(arr["offsets"][e], arr["offsets"][e + 1]):
                x = o.features(e, int(arr["q_idx"][r]), int(arr["budget"][r]))
                z = _torch_mlp(o, cfg, W, b, x, lb)
                np.testing.assert_allclose(lg[r], z, rtol=1e-12, atol=1e-12)
        o.schedule(arr, act)


def test_features_closed_form():
    """Feature vector against its definition evaluated with numpy float32."""
    cfg = workload.configs.get("c0")
    o, (W, b, emb, cap, lb) = make_oracle(cfg, seed=2, Q=32)
    cnt = workload.gen.counts(cfg, 2)
    for t in range(20):
        arr = workload.gen.tick(cfg, 2, t, cnt[t], 32)
        o.tick(arr)
    s = o.state()
    M, Ed = cfg["M"], cfg["embed_dim"]
    f32 = np.float32
    B = cfg["budget_max"]
    x = o.features(0, 5, 77)
    np.testing.assert_array_equal(x[:Ed], emb[5].astype(np.float64))
    for m in range(M):
        c = max(int(s["cap"][0, m]), 1)
        exp = [f32(s["qlen"][0, m]) * f32(1.0 / cfg["qcap"]),
               f32(s["busy"][0, m]) * f32(1.0 / c),
               f32(s["ewma"][0, m]) * f32(1.0 / (256.0 * B)),
               f32(s["backlog"][0, m]) * f32(1.0 / (c * B))]
        for k in range(4):
            assert x[Ed + k * M + m] == float(exp[k]), (m, k)
    assert x[Ed + 4 * M] == float(f32(77) * f32(1.0 / B))
    assert np.all(x[Ed + 4 * M + 1:] == 0.0)
