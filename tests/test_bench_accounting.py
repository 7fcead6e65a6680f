"""The benchmark's algorithmic work counts (the numerators of its roofline)
against the shapes of the generated policy and embedding table: per request
the layer-1 columns of its own features (embedding and budget; the load
statistics are shared by the env's requests, the pad column is zero) and
every later layer; per env the load-statistics columns; per request the
bytes of its record, its embedding row (element size of the table) and its
action."""
import numpy as np
import pytest

import bench
import workload

MLP = ["c0", "c1", "c2", "c3", "c4", "c2c"]


@pytest.mark.parametrize("name", MLP)
@pytest.mark.parametrize("value_head", [False, True])
def test_mlp_flops_from_weight_shapes(name, value_head):
    cfg = workload.configs.get(name, value_head=value_head)
    W, _ = workload.gen.weights(cfg, 0)
    H1, D = W[0].shape
    own = cfg["embed_dim"] + 1            # embedding | budget
    stats = 4 * cfg["M"]
    assert D >= own + stats               # the rest of the input row is zero padding
    assert W[-1].shape[0] == cfg["A"] + (1 if value_head else 0)
    per_req = H1 * own + sum(w.shape[0] * w.shape[1] for w in W[1:])
    per_env = H1 * stats
    for n in (0, 1, 262_142):
        assert bench.algorithmic_flops_per_tick(cfg, n) == 2 * (per_req * n + per_env * cfg["E"])


def test_dual_flops_from_weight_shapes():
    cfg = workload.configs.get("c2d", value_head=True)
    P = workload.gen.dual_weights(cfg, 0)
    shapes = {k: np.asarray(v).shape for k, v in P.items()}
    Ed = cfg["embed_dim"]
    # semantic layer over [query | role]: only its query half runs per request
    sem_out, sem_in = shapes["W_sem"]
    assert sem_in == 2 * Ed
    per_req = sem_out * Ed
    per_env = 0
    for k, v in shapes.items():
        if k in ("W_sem",) or not k.startswith("W_") or len(v) != 2:
            continue
        if k == "W_sys":                   # system head over 3 statistics per model: once per env
            per_env += v[0] * v[1]
        elif k == "W_res":                 # resource layer over [budget head | system head]
            half = v[1] // 2
            per_req += v[0] * half
            per_env += v[0] * (v[1] - half)
        else:
            per_req += v[0] * v[1]
    for n in (1, 262_142):
        assert bench.algorithmic_flops_per_tick(cfg, n) == 2 * (per_req * n + per_env * cfg["E"])


@pytest.mark.parametrize("name", MLP + ["c2d"])
@pytest.mark.parametrize("sample", [False, True])
def test_route_bytes_from_table(name, sample):
    cfg = workload.configs.get(name)
    table, _ = workload.gen.embedding(cfg, 0, rows=8)
    row = table.shape[1] * table.dtype.itemsize
    assert table.shape[1] == cfg["embed_dim"]
    rec = 4 + 2 + (2 if cfg.get("net") == "dual" else 0)   # q_idx int32, budget int16, role int16
    out = 4 + (12 if sample else 0)                         # action; log-prob, entropy, value fp32
    snap = 4 * 4 * cfg["M"] + cfg["M"]                      # per env: 4M fp32 statistics, M validity bytes
    n = 1000
    assert bench.algorithmic_bytes_route(cfg, n, sample) == (rec + row + out) * n + snap * cfg["E"]
