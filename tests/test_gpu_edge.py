"""GPU edge cases against the oracle: empty ticks, envs at the arrival limit,
invalid inputs (sticky error, env untouched), host knobs mid-run, state
checkpoint/resume, determinism, and exhaustive forced actions on tiny pools."""
import itertools

import numpy as np
import pytest

import oracle
import workload
from gpu_util import Pair, need_gpu, note
from helpers import assert_state_equal, check_invariants, tiny_cfg

pytestmark = pytest.mark.gpu


def _empty_tick(E):
    return dict(offsets=np.zeros(E + 1, np.int32), q_idx=np.zeros(0, np.int32),
                budget=np.zeros(0, np.int16), base_svc=np.zeros(0, np.int16))


def test_empty_ticks_and_drain():
    cfg = workload.configs.get("c1", E=6, T=30)
    note("[empty_ticks]")
    p = Pair(cfg, seed=21, Q=128)
    for t in range(30):
        arr = p.arrivals(t) if t < 10 else _empty_tick(cfg["E"])
        p.step(arr, mode="tick" if t % 2 else "route+schedule")
    p.compare_state(ctx="drain")
    p.close()


def test_arrival_limit_and_overflow():
    """An env exactly at max_arrivals is served; one above it is rejected with
    IM_ERR_COUNT and left untouched; a tiny queue overflows (tail-drop)."""
    cfg = workload.configs.get("c4", E=4, T=6, max_arrivals=100, qcap=40)
    note("[arrival_limit]")
    p = Pair(cfg, seed=22, Q=128)
    rng = np.random.default_rng(0)
    for t in range(6):
        counts = np.array([100, 0, 37, 101 if t == 3 else 5], np.int32)
        off = np.zeros(5, np.int32)
        off[1:] = np.cumsum(counts)
        n = int(off[-1])
        arr = dict(offsets=off, q_idx=rng.integers(0, 128, n).astype(np.int32),
                   budget=rng.integers(20, 400, n).astype(np.int16),
                   base_svc=rng.integers(1, 8, n).astype(np.int16))
        p.step(arr)
        p.compare_state(ctx=f"t={t}")
    assert p.gpu.error() & 2 and p.orc.error & 2
    s = p.gpu.state()
    assert s["rej_overflow"].sum() > 0
    p.close()


@pytest.mark.parametrize("what,bit", [("q_idx", 1), ("budget", 4), ("base_svc", 8),
                                      ("action", 16)])
def test_invalid_input_env_untouched(what, bit):
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c1", E=3, T=12)
    note(f"[invalid_input] {what}")
    p = Pair(cfg, seed=23, Q=64)
    for t in range(8):
        p.step(p.arrivals(t))
    arr = p.arrivals(8)
    lo, hi = int(arr["offsets"][1]), int(arr["offsets"][2])
    assert hi > lo
    before = p.gpu.state()
    dev0 = P.device_arrivals(arr)
    act = torch.zeros(len(arr["q_idx"]), dtype=torch.int32, device="cuda")
    p.gpu.route(dev0, act)
    if what == "q_idx":
        arr["q_idx"][lo] = 64
    elif what == "budget":
        arr["budget"][lo] = 0
    elif what == "base_svc":
        arr["base_svc"][lo] = 4096
    dev = P.device_arrivals(arr)
    if what == "action":
        act[lo] = cfg["A"]
    if what == "q_idx":
        p.gpu.route(dev, act)
        torch.cuda.synchronize()
        assert int(act[lo].item()) == -1
    p.gpu.clear_error()
    p.gpu.schedule(dev, act)
    assert p.gpu.error() & bit
    after = p.gpu.state()
    for k in ("next_id", "arrived", "qlen", "busy", "completed", "hist", "slots", "queues"):
        assert np.array_equal(np.asarray(before[k])[1], np.asarray(after[k])[1]), k
    # the other envs proceed exactly as the oracle says
    o_sub = dict(arr)
    p.orc.schedule(o_sub, act.cpu().numpy())
    assert p.orc.error & bit
    assert_state_equal(p.gpu.state(), p.orc.state(), ctx="after invalid env")
    p.close()


def test_host_knobs_midrun():
    cfg = workload.configs.get("c0", T=80)
    note("[host_knobs]")
    p = Pair(cfg, seed=24, Q=64)
    for t in range(80):
        if t == 15:
            p.gpu.set_enabled(0, 1, 0)
            p.orc.set_enabled(0, 1, 0)
            p.gpu.set_capacity(0, 2, 0)
            p.orc.set_capacity(0, 2, 0)
        if t == 50:
            p.gpu.set_enabled(0, 1, 1)
            p.orc.set_enabled(0, 1, 1)
            p.gpu.set_capacity(0, 2, 3)
            p.orc.set_capacity(0, 2, 3)
        act = p.step(p.arrivals(t))
        if 15 <= t < 50:
            assert not np.any((act // cfg["K"] == 1) | (act // cfg["K"] == 2))
        p.compare_state(ctx=f"t={t}")
    p.close()


def test_all_models_disabled_rejects():
    cfg = workload.configs.get("c1", E=2, T=5)
    p = Pair(cfg, seed=25, Q=64)
    for m in range(cfg["M"]):
        p.gpu.set_enabled(1, m, 0)
        p.orc.set_enabled(1, m, 0)
    for t in range(5):
        act = p.step(p.arrivals(t))
    s = p.compare_state(ctx="disabled")
    assert s["arrived"][1] == s["rej_nomodel"][1] > 0
    p.close()


def test_checkpoint_resume_equals_uninterrupted():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2", E=24, T=60, lam=16.0)
    note("[checkpoint]")
    a = Pair(cfg, seed=26, Q=256)
    for t in range(30):
        a.step(a.arrivals(t), mode="tick")
    snap = a.gpu.state()
    b = Pair(cfg, seed=26, Q=256)
    b.gpu.write_state(0, snap)
    assert_state_equal(b.gpu.state(), snap, ctx="round trip")
    for t in range(30, 60):
        arr = a.arrivals(t)
        dev = P.device_arrivals(arr)
        for q in (a, b):
            act = torch.zeros(max(len(arr["q_idx"]), 1), dtype=torch.int32, device="cuda")
            q.gpu.tick(dev, act)
    assert_state_equal(a.gpu.state(), b.gpu.state(), ctx="resume")
    a.close()
    b.close()


def test_write_state_rejects_inconsistent_entries():
    """A queued entry whose key is not the key mode's function of its arrival
    tick, budget and service time, or whose arrival tick is not before the
    snapshot's tick, is IM_ESTATE (the schedule step recovers arrival ticks
    from keys); nothing changes."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2", E=4, T=12, lam=16.0)
    p = Pair(cfg, seed=28, Q=128)
    for t in range(10):
        p.step(p.arrivals(t))
    snap = p.gpu.state()
    e, m = np.argwhere(snap["qlen"] > 0)[0]
    for field, delta in ((0, 1), (2, 1), (4, 1), (2, 10**6)):    # key, t_arr, budget, t_arr >= tick
        s2 = {k: np.array(v) for k, v in snap.items()}
        s2["queues"][e, m, 0, field] += delta
        with pytest.raises(P.IMError) as ei:
            p.gpu.write_state(0, s2)
        assert ei.value.status == P._lib.IM_ESTATE, (field, delta)
    assert_state_equal(p.gpu.state(), snap, ctx="unchanged")
    p.close()


def test_determinism_two_runs():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c3", E=64, T=40)
    note("[determinism]")
    runs = []
    for _ in range(2):
        p = Pair(cfg, seed=27, Q=256, e0=0, e1=1)
        for t in range(40):
            dev = P.device_arrivals(p.arrivals(t))
            p.gpu.tick(dev)
        runs.append(p.gpu.state())
        p.close()
    assert_state_equal(runs[0], runs[1], ctx="determinism")


def test_forced_actions_exhaustive():
    """Every forced-action vector over 4 arrivals on a tiny pool (M=2, K=2,
    QCAP=2, c=(1,2)): one GPU env per vector, all checked against the oracle."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    vecs = list(itertools.product(range(-1, 4), repeat=4))
    E = len(vecs)
    cfg = tiny_cfg(M=2, K=2, qcap=2, cap_hi=2, E=E, embed_dim=8, widths=[32, 4])
    note(f"[forced_actions] E={E}")
    W, b = workload.gen.weights(cfg, 0, 0.1)
    emb = np.zeros((4, 8), np.float32)
    cap = np.tile(np.array([[1, 2]], np.int32), (E, 1))
    gpu = P.Pool(cfg, W, b, torch.from_numpy(emb).cuda(), cap)
    orc = oracle.Oracle(cfg, W, b, emb, cap)
    rng = np.random.default_rng(5)
    hist = [[(int(rng.integers(1, 12)), int(rng.integers(1, 4)), int(rng.integers(-1, 4)))
             for _ in range(int(rng.integers(0, 4)))] for _ in range(3)]
    fields = [(int(rng.integers(1, 12)), int(rng.integers(1, 4))) for _ in range(4)]
    ticks = [[h] * E for h in hist]
    ticks.append([[(f[0], f[1], a) for f, a in zip(fields, v)] for v in vecs])
    ticks += [[[(5, 1, 0)]] * E, [[]] * E, [[]] * E]
    for ti, per_env in enumerate(ticks):
        counts = np.array([len(r) for r in per_env], np.int32)
        off = np.zeros(E + 1, np.int32)
        off[1:] = np.cumsum(counts)
        flat = [x for r in per_env for x in r]
        arr = dict(offsets=off, q_idx=np.zeros(len(flat), np.int32),
                   budget=np.array([x[0] for x in flat], np.int16),
                   base_svc=np.array([x[1] for x in flat], np.int16))
        acts = np.array([x[2] for x in flat], np.int32)
        dev = P.device_arrivals(arr)
        gpu.schedule(dev, torch.from_numpy(acts if acts.size else np.zeros(1, np.int32)).cuda())
        orc.schedule(arr, acts)
        s = gpu.state()
        assert_state_equal(s, orc.state(), ctx=f"tick {ti}")
        check_invariants(s, cfg, ctx=f"tick {ti}")
    assert gpu.error() == 0
    gpu.close()


def test_bf16_hidden_rounding_matches_rne():
    """The device's fp32 -> bf16 rounding of hidden activations, pinned to
    round-to-nearest-even: with 0/1 selection weights each logit equals one
    rounded hidden unit bf16(emb_a + b1_a), whose fp32 pre-image is known."""
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = tiny_cfg(M=4, K=8, qcap=8, cap_hi=1, embed_dim=32, widths=[32, 32], dtype="bf16",
                   E=1, max_arrivals=512)
    A, Ed, D = cfg["A"], 32, cfg["feat_dim"]
    rng = np.random.default_rng(9)
    W1 = np.zeros((32, D), np.float32)
    W1[np.arange(32), np.arange(32)] = 1.0
    W2 = np.eye(32, dtype=np.float32)
    b2 = np.zeros(32, np.float32)
    # embedding values (bf16) in [1, 2) and fp32 biases with low mantissa bits
    # set, so the sums exercise ties and both rounding directions
    Q = 512
    emb_f = (1.0 + rng.integers(0, 128, (Q, Ed)) / 128.0).astype(np.float32)
    emb_bits = torch.from_numpy(emb_f).to(torch.bfloat16).view(torch.int16).numpy()
    b1 = (rng.integers(0, 1 << 16, 32) * 2.0 ** -23).astype(np.float32)
    b1[:4] = [2.0 ** -9, 3 * 2.0 ** -9, 2.0 ** -8, 2.0 ** -9 + 2.0 ** -20]
    pool = P.Pool(cfg, [W1, W2], [b1, b2], torch.from_numpy(emb_bits).cuda(),
                  np.ones((1, cfg["M"]), np.int32))
    n = Q
    arr = dict(offsets=np.array([0, n], np.int32), q_idx=np.arange(n, dtype=np.int32),
               budget=np.full(n, 5, np.int16), base_svc=np.ones(n, np.int16))
    dev = P.device_arrivals(arr)
    act = torch.zeros(n, dtype=torch.int32, device="cuda")
    lg = torch.zeros((n, A), dtype=torch.float32, device="cuda")
    pool.route(dev, act, lg)
    torch.cuda.synchronize()
    got = lg.cpu().numpy().astype(np.float64)
    pre = (emb_f + b1[None, :]).astype(np.float32)          # fp32 sums, RNE
    exp = oracle.round_bf16_array(np.maximum(pre, 0).astype(np.float64))
    np.testing.assert_array_equal(got, exp)
    pool.close()
