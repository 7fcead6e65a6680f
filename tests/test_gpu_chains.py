"""GPU parity of multi-step agent chains (Sec. 4.3, pools with max_steps > 1)
against the oracle.

Lockstep per tick through the rows the device builds (each env's pending
calls, then its arrivals): logits within the tolerance, actions equal except
at near-ties, and the whole state bit-exact, including every queued call's and
slot's chain words, the pending calls with their inherited deadlines and the
query counters. Also: im_tick, every key mode, RL rollouts, the dual-pathway
executor with rotating roles, the full-size pool in the benchmark's launch
configuration on sampled envs, ticks replayed from a captured graph whose
length is odd (the pending buffers alternate by tick parity on the device),
the dual update over queries, bad n_steps and the rejected calls."""
import numpy as np
import pytest

import oracle
import workload
from gpu_util import Pair, need_gpu, note

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["slack", "deadline", "fcfs"])
def test_chain_lockstep(mode):
    cfg = workload.configs.get("c2c", E=16, T=40, key_mode=mode, lam=6.0, qcap=128)
    note(f"[chain_lockstep] c2c E=16 mode={mode}")
    p = Pair(cfg, seed=41, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t), mode="tick" if t % 3 == 2 else "route+schedule")
        if t % 5 == 4:
            p.compare_state(ctx=f"{mode} t={t}")
    s = p.compare_state(ctx="end")
    assert s["q_done"].sum() > 100
    note(f"  rows={p.rows_checked} flips={p.flips} queries done={int(s['q_done'].sum())}")
    assert p.gpu.error() == 0
    p.close()


def test_chain_heavy_load_overflow():
    """lambda = 16 queries of up to 4 calls into small queues: tail drops end
    queries, late calls carry budgets <= 0."""
    cfg = workload.configs.get("c2c", E=12, T=40, qcap=32, budget_lo=5, budget_hi=60)
    note("[chain_heavy] c2c E=12 qcap=32")
    p = Pair(cfg, seed=42, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
    s = p.compare_state(ctx="end")
    assert s["rej_overflow"].sum() > 0
    gc = p.gpu.chain_state()
    valid = np.arange(gc["pending"].shape[1])[None, :] < gc["pending_count"][:, None]
    late = valid & (gc["pending"][..., 6] < cfg["T"])
    note(f"  overflow={int(s['rej_overflow'].sum())} pending past deadline={int(late.sum())}")
    p.close()


def test_chain_rl_lockstep():
    cfg = workload.configs.get("c2c", E=8, T=25, value_head=True, lam=6.0)
    note("[chain_rl] c2c E=8 value head")
    p = Pair(cfg, seed=43, Q=256)
    for t in range(cfg["T"]):
        p.step_rl(p.arrivals(t), seed=0xC4A1 + t)
        if t % 6 == 5:
            p.compare_state(ctx=f"rl t={t}")
    p.close()


def test_chain_dual_executor():
    cfg = workload.configs.get("c2d", E=12, T=25, embed_dim=64, max_steps=4, lam=8.0)
    note("[chain_dual] c2d E_d=64 max_steps=4")
    p = Pair(cfg, seed=44, Q=256)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 6 == 5:
            p.compare_state(ctx=f"dual t={t}")
    p.close()


def test_chain_full_size_sampled():
    cfg = workload.configs.get("c2c", T=14)
    note(f"[chain_full_size] c2c E={cfg['E']} envs [1000,1004)")
    p = Pair(cfg, seed=0, e0=1000, e1=1004)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t), check_logits=(t % 4 == 0))
    p.compare_state(ctx="full size")
    note(f"  rows={p.rows_checked} flips={p.flips}")
    assert p.gpu.error() == 0
    p.close()


def test_chain_graph_replay_odd_length():
    """Three ticks captured once, replayed twice: the device picks the pending
    buffers by the tick it holds, so the replays continue the chains."""
    torch = need_gpu()
    cfg = workload.configs.get("c2c", E=8, T=12, lam=6.0)
    note("[chain_graph] c2c E=8 3-tick graph x2")
    p = Pair(cfg, seed=45, Q=256)
    for t in range(3):
        p.step(p.arrivals(t))
    arrs = [p.arrivals(t) for t in range(3, 6)]
    devs = [p.P.device_arrivals(a) for a in arrs]
    n = max(p._rows(a) for a in arrs)
    act = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            for d in devs:
                p.gpu.tick(d, act)
    torch.cuda.synchronize()
    # capture does not run the ticks; the oracle runs the same arrivals twice
    for rep in range(2):
        g.replay()
        torch.cuda.synchronize()
        for a in arrs:
            p.orc.tick(workload.gen.subset(a, p.e0, p.e1))
        p.compare_state(ctx=f"replay {rep}")
    assert p.gpu.error() == 0
    p.close()


def test_chain_dual_update_counts_queries():
    torch = need_gpu()
    cfg = workload.configs.get("c2c", E=6, T=30, lam=4.0)
    note("[chain_dual_update] c2c E=6")
    p = Pair(cfg, seed=46, Q=128)
    lam = torch.tensor([0.5], dtype=torch.float64, device="cuda")
    lo = 0.5
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 5 == 4:
            p.gpu.dual_update(0.25, 4.0, lam)
            torch.cuda.synchronize()
            lo = p.orc.dual_update(lo, 0.25, 4.0)
            assert float(lam.cpu()[0]) == lo, (t, float(lam.cpu()[0]), lo)
    assert lo != 0.5
    p.close()


def test_chain_bad_n_steps_env_untouched():
    torch = need_gpu()
    cfg = workload.configs.get("c2c", E=4, T=10, lam=6.0)
    note("[chain_bad_steps] c2c E=4")
    p = Pair(cfg, seed=47, Q=128)
    for t in range(6):
        p.step(p.arrivals(t))
    arr = workload.gen.tick(cfg, 47, 6, np.array([2, 3, 1, 2], np.int32), p.Q)
    arr["n_steps"] = arr["n_steps"].copy()
    arr["n_steps"][3] = cfg["max_steps"] + 1          # env 1
    arr["n_steps"][5] = 0                            # env 2
    before, chb = p.gpu.state(), p.gpu.chain_state()
    p.step(arr, check_logits=False)
    assert p.gpu.error() & oracle.ERR_STEPS and p.orc.error & oracle.ERR_STEPS
    after, cha = p.gpu.state(), p.gpu.chain_state()
    for e in (1, 2):
        for k in ("qlen", "enqueued", "started", "completed"):
            np.testing.assert_array_equal(after[k][e], before[k][e], err_msg=f"{k} env {e}")
        assert cha["pending_count"][e] == chb["pending_count"][e]
        np.testing.assert_array_equal(cha["pending"][e], chb["pending"][e])
    p.compare_state(ctx="bad n_steps")
    # the kept pending calls are routed at the next tick
    p.gpu.clear_error()
    p.orc.clear_error()
    p.step(p.arrivals(7))
    p.compare_state(ctx="after")
    p.close()


def test_chain_pool_refuses_missing_n_steps_and_write_state():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2c", E=2, T=3)
    p = Pair(cfg, seed=48, Q=64)
    arr = p.arrivals(0)
    del arr["n_steps"]
    dev = P.device_arrivals(arr)
    act = torch.zeros(p._rows(p.arrivals(0)), dtype=torch.int32, device="cuda")
    with pytest.raises(P.IMError) as ei:
        p.gpu.route(dev, act)
    assert ei.value.status == P._lib.IM_EINVAL
    s = p.gpu.state()
    with pytest.raises(P.IMError) as ei:
        p.gpu.write_state(0, s)
    assert ei.value.status == P._lib.IM_EUNSUPPORTED
    p.close()
