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
from helpers import assert_state_equal
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


@pytest.mark.timeout(600)
def test_chain_full_size_sampled():
    cfg = workload.configs.get("c2c", T=64)
    note(f"[chain_full_size] c2c E={cfg['E']} T={cfg['T']} envs [1000,1004)")
    p = Pair(cfg, seed=0, e0=1000, e1=1004)
    for t in range(cfg["T"]):
        p.step(p.arrivals(t), check_logits=(t % 8 == 0))
        if t % 16 == 15:
            p.compare_state(ctx=f"full size t={t}")
            note(f"  t={t} ok")
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


def test_chain_broken_csr_skips_every_env():
    """Offsets that are not one monotone partition of [0, n_total) (env 2
    re-reads env 0's records) in a chain pool: no arrival is routed, every env
    skips the tick with IM_ERR_COUNT and keeps its pending calls, bit-exact
    with the oracle; nothing is written past the caller's row buffers (sized
    n_total + E*M*S), and the kept calls are routed at the next tick."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2c", E=3, T=10, lam=6.0)
    note("[chain_broken_csr] c2c E=3")
    p = Pair(cfg, seed=49, Q=128)
    for t in range(6):
        p.step(p.arrivals(t))
    arr = workload.gen.tick(cfg, 49, 6, np.array([20, 2, 2], np.int32), p.Q)
    arr["offsets"] = np.array([0, 20, 2, 24], np.int32)
    n = p._rows(arr)
    guard = 4096
    act = torch.full((n + guard,), -7, dtype=torch.int32, device="cuda")
    lg = torch.full((n + guard, cfg["A"]), 7.0, dtype=torch.float32, device="cuda")
    dev = P.device_arrivals(arr)
    chb = p.gpu.chain_state()
    p.gpu.route(dev, act, lg)
    torch.cuda.synchronize()
    off, nrows = p.gpu.rows()
    assert nrows == int(chb["pending_count"].sum())
    assert bool((act[n:] == -7).all()) and bool((lg[n:] == 7.0).all())
    sub = workload.gen.subset(arr, 0, cfg["E"])
    o_act, _ = p.orc.route(sub)
    assert int(p.orc.row_offsets(sub)[-1]) == nrows      # the oracle's rows: pending calls only
    g_act = act[:nrows].cpu().numpy()
    for r in np.nonzero(g_act != o_act[:nrows])[0]:
        assert g_act[r] >= 0 and o_act[r] >= 0, r       # near ties only (checked with logits elsewhere)
    p.gpu.schedule(dev, act)
    p.orc.schedule(sub, act[:nrows].cpu().numpy())
    torch.cuda.synchronize()
    assert p.gpu.error() & oracle.ERR_COUNT and p.orc.error & oracle.ERR_COUNT
    cha = p.gpu.chain_state()
    np.testing.assert_array_equal(cha["pending_count"], chb["pending_count"])
    p.compare_state(ctx="broken csr")
    p.gpu.clear_error()
    p.orc.clear_error()
    p.step(p.arrivals(7))
    p.compare_state(ctx="after")
    assert p.gpu.error() == 0
    p.close()


def _chain_eq(x, y, ctx):
    for k in ("queue_chain", "slot_chain", "pending", "pending_count"):
        np.testing.assert_array_equal(x[k], y[k], err_msg=f"{ctx}: {k}")


def test_chain_checkpoint_resume():
    """im_write_chain_state: a chain pool run for 20 ticks, snapshot (state,
    chain words of queued and running calls, pending calls) written into a
    fresh pool; both pools then run 20 more ticks. The resumed pool equals the
    uninterrupted one bit for bit, which stays in lockstep with the oracle."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2c", E=8, T=40, lam=8.0, qcap=256)
    note("[chain_checkpoint] c2c E=8")
    a = Pair(cfg, seed=50, Q=256)
    for t in range(20):
        a.step(a.arrivals(t), mode="tick" if t % 2 else "route+schedule")
    snap, ch = a.gpu.state(), a.gpu.chain_state()
    assert ch["pending_count"].sum() > 0 and (ch["queue_chain"][..., 2] > 1).any()
    b = Pair(cfg, seed=50, Q=256)
    b.gpu.write_chain_state(0, snap, ch)
    assert_state_equal(b.gpu.state(), snap, ctx="round trip")
    _chain_eq(b.gpu.chain_state(), ch, "round trip")
    for t in range(20, 40):
        arr = a.arrivals(t)
        a.step(arr)
        b.gpu.tick(P.device_arrivals(arr))
    a.compare_state(ctx="uninterrupted vs oracle")
    assert_state_equal(b.gpu.state(), a.gpu.state(), ctx="resumed vs uninterrupted")
    _chain_eq(b.gpu.chain_state(), a.gpu.chain_state(), "resumed vs uninterrupted")
    assert a.gpu.error() == 0 and b.gpu.error() == 0
    a.close()
    b.close()


def test_chain_write_state_rejects_bad_chain_words():
    """A chain word out of range (call index past its query's calls, a
    pending call numbered 0, a base service time not dividing the queued
    service time) is IM_ESTATE and changes nothing."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2c", E=4, T=12, lam=8.0)
    p = Pair(cfg, seed=51, Q=128)
    for t in range(10):
        p.step(p.arrivals(t))
    snap, ch = p.gpu.state(), p.gpu.chain_state()
    e, m = np.argwhere(snap["qlen"] > 0)[0]
    bad = []
    c1 = {k: np.array(v) for k, v in ch.items()}
    c1["queue_chain"][e, m, 0, 1] = c1["queue_chain"][e, m, 0, 2]          # k = n_steps
    bad.append(c1)
    c2 = {k: np.array(v) for k, v in ch.items()}
    c2["queue_chain"][e, m, 0, 4] = int(snap["queues"][e, m, 0, 3]) + 1    # base_svc > svc
    bad.append(c2)
    ep = int(np.argmax(ch["pending_count"]))
    if ch["pending_count"][ep] > 0:
        c3 = {k: np.array(v) for k, v in ch.items()}
        c3["pending"][ep, 0, 1] = 0                                        # pending call k = 0
        bad.append(c3)
    for c in bad:
        with pytest.raises(P.IMError) as ei:
            p.gpu.write_chain_state(0, snap, c)
        assert ei.value.status == P._lib.IM_ESTATE
    assert_state_equal(p.gpu.state(), snap, ctx="unchanged")
    _chain_eq(p.gpu.chain_state(), ch, "unchanged")
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
