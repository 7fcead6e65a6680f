"""GPU parity of the RL-rollout route (im_route_sample) against the oracle.

Lockstep per tick on every workload with a value head: logits within the
tolerance (1e-4 fp32, 2e-2 bf16, relative to the row's largest logit), sampled
actions equal except where the oracle's perturbed scores of the two actions
are within twice that tolerance, log-probs / entropies / values within the
tolerance they inherit from the logits, and the integer state after
im_schedule with those actions bit-exact. Also: greedy mode equals im_route,
the full-size c2 pool in the benchmark's launch configuration on sampled
envs, the sample distribution of the GPU against its own softmax (a property
that holds at any size), and the edge cases."""
import numpy as np
import pytest
import scipy.special
import scipy.stats

import workload
from gpu_util import Pair, need_gpu, note

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,E,T", [("c0", 1, 60), ("c1", 8, 25), ("c2", 8, 30),
                                      ("c3", 3, 20), ("c4", 12, 25)])
def test_rl_lockstep_small(name, E, T):
    cfg = workload.configs.get(name, E=E, T=T, value_head=True)
    note(f"[rl_lockstep_small] {name} E={E} T={T}")
    p = Pair(cfg, seed=21, Q=512)
    for t in range(T):
        p.step_rl(p.arrivals(t), seed=0x5EED0000 + t)
        if t % 5 == 4:
            p.compare_state(ctx=f"{name} t={t}")
    note(f"  rows={p.rows_checked} near-tie flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()


def test_rl_greedy_is_route():
    torch = need_gpu()
    cfg = workload.configs.get("c2", E=16, T=20, value_head=True)
    note("[rl_greedy_is_route] c2 E=16")
    p = Pair(cfg, seed=22, Q=512)
    for t in range(cfg["T"]):
        arr = p.arrivals(t)
        dev = p.P.device_arrivals(arr)
        n = max(int(arr["q_idx"].size), 1)
        a_route = torch.empty(n, dtype=torch.int32, device="cuda")
        p.gpu.route(dev, a_route)
        torch.cuda.synchronize()
        a_greedy = p.step_rl(arr, seed=5, greedy=True)
        np.testing.assert_array_equal(a_greedy, a_route.cpu().numpy()[:a_greedy.size])
    p.compare_state(ctx="greedy end")
    p.close()


def test_rl_full_size_sampled():
    cfg = workload.configs.get("c2", T=40, value_head=True)
    note(f"[rl_full_size] c2 E={cfg['E']} T={cfg['T']} envs [2000,2005)")
    p = Pair(cfg, seed=0, e0=2000, e1=2005)
    for t in range(cfg["T"]):
        p.step_rl(p.arrivals(t), seed=77 + t)
        if t % 10 == 9:
            p.compare_state(ctx=f"c2 full t={t}")
            note(f"  t={t} ok")
    assert p.gpu.error() == 0
    p.close()


def test_rl_sample_distribution():
    """Many identical requests in one env: the GPU's sampled actions follow
    the softmax of its own logits over the valid actions (chi-square)."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    from helpers import tiny_cfg
    n = 60000
    cfg = tiny_cfg(M=3, K=3, widths=[32, 9], max_arrivals=n, qcap=8, value_head=True)
    W, b = workload.gen.weights(cfg, 4, 0.5)
    table, _ = workload.gen.embedding(cfg, 4, rows=8)
    pool = P.Pool(cfg, W, b, torch.from_numpy(table).cuda(), np.full((1, 3), 2, np.int32))
    pool.set_enabled(0, 1, 0)
    arr = dict(offsets=np.array([0, n], np.int32), q_idx=np.full(n, 3, np.int32),
               budget=np.full(n, 50, np.int16), base_svc=np.ones(n, np.int16))
    dev = P.device_arrivals(arr)
    act = torch.empty(n, dtype=torch.int32, device="cuda")
    lg = torch.empty((n, 9), dtype=torch.float32, device="cuda")
    lp = torch.empty(n, dtype=torch.float32, device="cuda")
    pool.route_sample(dev, 0xABCDEF0123, act, lp, None, None, lg)
    torch.cuda.synchronize()
    z = lg[0].cpu().numpy().astype(np.float64)
    assert np.all(lg.cpu().numpy() == lg[0].cpu().numpy())
    valid = np.array([a // 3 != 1 for a in range(9)])
    p = np.zeros(9)
    p[valid] = scipy.special.softmax(z[valid])
    counts = np.bincount(act.cpu().numpy(), minlength=9)
    assert counts[~valid].sum() == 0
    stat = ((counts[valid] - n * p[valid]) ** 2 / (n * p[valid])).sum()
    assert scipy.stats.chi2.sf(stat, valid.sum() - 1) > 1e-4, (counts, n * p)
    np.testing.assert_allclose(lp.cpu().numpy(), np.log(p[act.cpu().numpy()]), atol=1e-5)
    pool.close()


def test_rl_edge_cases():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    from helpers import tiny_cfg
    cfg = tiny_cfg(M=2, K=2, widths=[32, 4], value_head=True)
    W, b = workload.gen.weights(cfg, 9, 0.1)
    table, _ = workload.gen.embedding(cfg, 9, rows=8)
    pool = P.Pool(cfg, W, b, torch.from_numpy(table).cuda(), np.full((1, 2), 1, np.int32))
    pool.set_enabled(0, 0, 0)
    pool.set_enabled(0, 1, 0)
    arr = dict(offsets=np.array([0, 3], np.int32), q_idx=np.array([1, 2, 9], np.int32),
               budget=np.full(3, 5, np.int16), base_svc=np.ones(3, np.int16))
    dev = P.device_arrivals(arr)
    f = lambda: torch.full((3,), 7.0, dtype=torch.float32, device="cuda")  # noqa: E731
    act = torch.full((3,), 5, dtype=torch.int32, device="cuda")
    lp, en, va = f(), f(), f()
    pool.route_sample(dev, 1, act, lp, en, va)
    torch.cuda.synchronize()
    assert act.cpu().tolist() == [-1, -1, -1]             # nothing valid; row 2 has q_idx 9 >= Q
    assert lp.cpu().tolist() == [0, 0, 0] and en.cpu().tolist() == [0, 0, 0]
    v = va.cpu().numpy()
    assert v[0] != 0 and v[1] != 0 and v[2] == 0
    assert pool.error() == 1                              # IM_ERR_QIDX
    pool.clear_error()
    cfg2 = tiny_cfg(M=2, K=2, widths=[32, 4])
    W2, b2 = workload.gen.weights(cfg2, 9, 0.1)
    pool2 = P.Pool(cfg2, W2, b2, torch.from_numpy(table).cuda(), np.full((1, 2), 1, np.int32))
    with pytest.raises(P.IMError):
        pool2.route_sample(dev, 1, act, lp, en, va)      # no value head
    pool.close()
    pool2.close()
