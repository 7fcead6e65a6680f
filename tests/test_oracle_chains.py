"""Pins of the oracle's multi-step agent chains (Sec. 4.3: every call a query's
agents generate inherits the query's deadline t_arrive + beta).

* A three-call query through a one-slot model in closed form: the calls run
  back to back with one routing tick between them, each routed with the
  remaining budget deadline - t, the query completes on time, the cost is the
  sum over its calls of floor(2^16 latency / beta), the dual update (Eq. 7)
  counts it once.
* The remaining budget and the inherited query embedding reach the policy:
  a pending call's logits equal the MLP on features(q_idx, deadline - t).
* A chain pool whose queries all have one call is the single-step pool.
* An independent list model of chains (Python lists, sorted(), written from
  the rules above) against the oracle tick by tick under random forced
  actions on tiny pools, every key mode.
* Invariants on random chain workloads: call conservation, query
  conservation (arrived = completed + dropped + in flight), and on every
  queued or running call beta - budget >= k (call k is routed at least one
  tick after call k - 1 was, so at least k ticks after its query arrived).
* Bad n_steps: error bit, env untouched, its pending calls kept.
* Dual-pathway pools route call k with role (role_0 + k) mod n_roles.
"""
import numpy as np
import pytest

import oracle
import workload
from helpers import check_invariants, make_oracle


def _tiny_cfg(**kw):
    base = dict(E=1, M=1, K=1, cap_lo=1, cap_hi=1, qcap=16, widths=[32, 1], feat_dim=40,
                embed_dim=32, dtype="f32", key_mode="deadline", T=30, budget_hi=100)
    base.update(kw)
    return workload.configs.get("c2c", **base)


def _arr(q=(), budget=(), svc=(), steps=(), E=1, counts=None):
    counts = [len(q)] if counts is None else counts
    off = np.zeros(E + 1, np.int32)
    off[1:] = np.cumsum(counts)
    return dict(offsets=off, q_idx=np.array(q, np.int32), budget=np.array(budget, np.int16),
                base_svc=np.array(svc, np.int16), n_steps=np.array(steps, np.int16))


def _forced(o, arr, action_of_row):
    """Schedule one tick with the action `action_of_row(e, i)` for row i of env e."""
    ro = o.row_offsets(arr)
    act = np.full(max(int(ro[-1]), 1), -1, np.int32)
    for e in range(o.E):
        for i in range(int(ro[e + 1] - ro[e])):
            act[ro[e] + i] = action_of_row(e, i)
    o.schedule(arr, act)
    return act


def test_three_call_query_closed_form():
    cfg = _tiny_cfg()
    o, _ = make_oracle(cfg, seed=1, Q=8)
    empty = _arr()
    rows_per_tick = []
    for t in range(7):
        arr = _arr([3], [50], [2], [3]) if t == 0 else empty
        ro = o.row_offsets(arr)
        rows_per_tick.append(int(ro[-1]))
        if t in (2, 4):
            ch = o.chain_state()
            assert ch["pending_count"][0] == 1
            q_idx, k, n, role0, base, beta, dl = ch["pending"][0, 0]
            assert (q_idx, k, n, base, beta, dl) == (3, t // 2, 3, 2, 50, 50)
        _forced(o, arr, lambda e, i: 0)
        s = o.state()
        if t in (0, 2, 4):
            # the call entered its slot at t (t_arr = t) with budget 50 - t
            sl = s["slots"][0, 0, 0]
            assert tuple(sl) == (t // 2, t, 2 - 1, 50 - t), (t, sl)
    assert rows_per_tick == [1, 0, 1, 0, 1, 0, 0]
    s, ch = o.state(), o.chain_state()
    assert s["completed"][0, 0] == 3 and s["lat_sum"][0, 0] == 6 and s["slo_met"][0, 0] == 3
    assert s["cost_q16"][0, 0] == 3 * ((2 << 16) // 50)
    assert ch["q_done"][0] == 1 and ch["q_met"][0] == 1 and ch["pending_count"][0] == 0
    assert s["next_id"][0] == 3 and s["arrived"][0] == 3
    lam = o.dual_update(1.0, 0.5, 10.0)
    cbar = 3 * ((2 << 16) // 50) / 65536.0
    assert lam == max(0.0, 1.0 + 0.5 * (cbar - 1.0))


def test_late_query_keeps_its_deadline():
    """A query whose budget runs out mid-chain: later calls are routed with a
    remaining budget <= 0 and the query completes late."""
    cfg = _tiny_cfg(key_mode="slack")
    o, _ = make_oracle(cfg, seed=2, Q=8)
    for t in range(12):
        arr = _arr([1], [3], [2], [4]) if t == 0 else _arr()
        if t == 4:
            ch = o.chain_state()
            assert ch["pending"][0, 0, 6] == 3          # deadline 0 + 3
        _forced(o, arr, lambda e, i: 0)
        if t == 4:
            sl = o.state()["slots"][0, 0, 0]
            assert sl[3] == 3 - 4                       # remaining budget -1
    ch = o.chain_state()
    assert ch["q_done"][0] == 1 and ch["q_met"][0] == 0
    s = o.state()
    assert s["completed"][0, 0] == 4 and s["slo_met"][0, 0] == 1   # only the first call on time


def _mlp64(cfg, W, b, x):
    h = np.asarray(x, np.float64)
    for l in range(len(W)):
        h = W[l].astype(np.float64) @ h + b[l].astype(np.float64)
        if l + 1 < len(W):
            h = np.maximum(h, 0.0)
    return h


def test_pending_call_sees_remaining_budget():
    cfg = workload.configs.get("c2c", E=3, T=20, dtype="f32")
    o, (W, b, emb, cap, lb) = make_oracle(cfg, seed=3, Q=64)
    cnt = workload.gen.counts(cfg, 3)
    checked = 0
    for t in range(20):
        arr = workload.gen.tick(cfg, 3, t, cnt[t], 64)
        ch = o.chain_state()
        ro = o.row_offsets(arr)
        act, lg = o.route(arr)
        for e in range(cfg["E"]):
            for i in range(int(ch["pending_count"][e])):
                q_idx, k, n, role0, base, beta, dl = ch["pending"][e, i]
                x = o.features(e, int(q_idx), int(dl) - t)
                z = _mlp64(cfg, W, b, x)
                np.testing.assert_allclose(lg[ro[e] + i], z, rtol=1e-12, atol=1e-12)
                checked += 1
        o.schedule(arr, act)
    assert checked > 20


def _steps(cfg, arr, value):
    a = dict(arr)
    a["n_steps"] = np.full(arr["q_idx"].size, value, np.int16)
    return a


def test_single_call_queries_equal_single_step_pool():
    cfg_c = workload.configs.get("c2c", E=4, T=25)
    cfg_s = workload.configs.get("c2c", E=4, T=25, max_steps=1)
    oc, _ = make_oracle(cfg_c, seed=4, Q=128)
    os_, _ = make_oracle(cfg_s, seed=4, Q=128)
    cnt = workload.gen.counts(cfg_c, 4)
    for t in range(cfg_c["T"]):
        arr = _steps(cfg_c, workload.gen.tick(cfg_c, 4, t, cnt[t], 128), 1)
        a1, l1 = oc.route(arr)
        a2, l2 = os_.route(arr)
        np.testing.assert_array_equal(a1, a2)
        np.testing.assert_array_equal(l1, l2)
        oc.schedule(arr, a1)
        os_.schedule(arr, a2)
    s1, s2 = oc.state(), os_.state()
    for k in ("qlen", "busy", "ewma", "completed", "slo_met", "cost_q16", "next_id", "queues", "slots"):
        np.testing.assert_array_equal(s1[k], s2[k], err_msg=k)
    assert oc.chain_state()["q_done"].sum() == s1["completed"].sum()


class ChainList:
    """Independent list model of one env with chains (tiny pools)."""

    def __init__(self, M, K, qcap, caps, key_mode):
        self.M, self.K, self.qcap, self.caps, self.mode = M, K, qcap, caps, key_mode
        self.t = 0
        self.next_id = 0
        self.q = [[] for _ in range(M)]
        self.slots = [[None] * max(caps) for _ in range(M)]
        self.pending = []
        self.ewma = [0] * M
        self.c = {k: [0] * M for k in ("rej_overflow", "enqueued", "started", "completed",
                                       "slo_met", "lat_sum", "wait_sum", "cost_q16")}
        self.q_done = self.q_met = 0

    def rows(self, arrivals):
        """arrivals: list of (q_idx, budget, base_svc, n_steps)."""
        out = [dict(q=p["q"], k=p["k"], n=p["n"], base=p["base"], beta=p["beta"],
                    budget=max(-32768, p["deadline"] - self.t)) for p in self.pending]
        out += [dict(q=q, k=0, n=n, base=s, beta=b, budget=b) for (q, b, s, n) in arrivals]
        return out

    def key(self, budget, svc):
        return {"deadline": self.t + budget, "fcfs": self.t}.get(self.mode, self.t + budget - svc)

    def step(self, arrivals, actions):
        rows = self.rows(arrivals)
        t = self.t
        for m in range(self.M):
            new = []
            for i, (r, a) in enumerate(zip(rows, actions)):
                if a < 0 or a // self.K != m:
                    continue
                if len(self.q[m]) + len(new) >= self.qcap:
                    self.c["rej_overflow"][m] += 1
                    continue
                svc = r["base"] * (a % self.K + 1)
                new.append(dict(r, key=self.key(r["budget"], svc), id=self.next_id + i, t_arr=t, svc=svc))
                self.c["enqueued"][m] += 1
            self.q[m] = sorted(self.q[m] + new, key=lambda x: (x["key"], x["id"]))
        spawned = []
        for m in range(self.M):
            for s in range(self.caps[m]):
                if self.slots[m][s] is None and self.q[m]:
                    x = self.q[m].pop(0)
                    self.slots[m][s] = dict(x, rem=x["svc"])
                    self.c["started"][m] += 1
                    self.c["wait_sum"][m] += t - x["t_arr"]
            for s in range(len(self.slots[m])):
                x = self.slots[m][s]
                if x is None:
                    continue
                x["rem"] -= 1
                if x["rem"]:
                    continue
                lat = t - x["t_arr"] + 1
                self.ewma[m] += (lat * 256 - self.ewma[m]) // 8
                self.c["completed"][m] += 1
                self.c["lat_sum"][m] += lat
                ok = lat <= x["budget"]
                self.c["slo_met"][m] += int(ok)
                self.c["cost_q16"][m] += (lat << 16) // x["beta"]
                if x["k"] + 1 < x["n"]:
                    spawned.append(dict(q=x["q"], k=x["k"] + 1, n=x["n"], base=x["base"],
                                        beta=x["beta"], deadline=x["t_arr"] + x["budget"]))
                else:
                    self.q_done += 1
                    self.q_met += int(ok)
                self.slots[m][s] = None
        self.pending = spawned
        self.next_id += len(rows)
        self.t += 1


@pytest.mark.parametrize("mode", ["slack", "deadline", "fcfs"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_chain_list_model(mode, seed):
    M, K, qcap = 2, 2, 4
    rng = np.random.default_rng(100 + seed)
    caps = [int(c) for c in rng.integers(1, 3, size=M)]
    cfg = workload.configs.get("c2c", E=1, M=M, K=K, qcap=qcap, cap_lo=1, cap_hi=2, key_mode=mode,
                               widths=[32, M * K], feat_dim=32 + 4 * M + 1, embed_dim=32, dtype="f32",
                               T=60, budget_hi=30)
    o, _ = make_oracle(cfg, seed=seed, Q=16, cap=np.array([caps], np.int32))
    ref = ChainList(M, K, qcap, caps, mode)
    for t in range(60):
        na = int(rng.integers(0, 3))
        arrivals = [(int(rng.integers(0, 16)), int(rng.integers(1, 31)), int(rng.integers(1, 4)),
                     int(rng.integers(1, 5))) for _ in range(na)]
        arr = _arr([a[0] for a in arrivals], [a[1] for a in arrivals], [a[2] for a in arrivals],
                   [a[3] for a in arrivals])
        nrows = len(ref.pending) + na
        assert int(o.row_offsets(arr)[-1]) == nrows
        acts = [int(rng.integers(-1, M * K)) for _ in range(nrows)]
        _forced(o, arr, lambda e, i: acts[i])
        ref.step(arrivals, acts)
        s, ch = o.state(), o.chain_state()
        for m in range(M):
            n = int(s["qlen"][0, m])
            got = [tuple(x) for x in s["queues"][0, m, :n]]
            exp = [(x["key"], x["id"], x["t_arr"], x["svc"], x["budget"]) for x in ref.q[m]]
            assert got == exp, (t, m)
            for k in ref.c:
                assert s[k][0, m] == ref.c[k][m], (t, m, k)
            assert s["ewma"][0, m] == ref.ewma[m]
        pend = [tuple(x) for x in ch["pending"][0, :ch["pending_count"][0]]]
        exp_p = [(p["q"], p["k"], p["n"], 0, p["base"], p["beta"], p["deadline"]) for p in ref.pending]
        assert pend == exp_p, t
        assert (ch["q_done"][0], ch["q_met"][0]) == (ref.q_done, ref.q_met)


@pytest.mark.parametrize("mode", ["slack", "deadline"])
def test_chain_invariants_random_workload(mode):
    cfg = workload.configs.get("c2c", E=6, T=60, key_mode=mode, lam=6.0, qcap=64)
    o, _ = make_oracle(cfg, seed=5, Q=128)
    cnt = workload.gen.counts(cfg, 5)
    queries = 0
    prev = None
    for t in range(cfg["T"]):
        arr = workload.gen.tick(cfg, 5, t, cnt[t], 128)
        queries += int(arr["q_idx"].size)
        o.tick(arr)
        s, ch = o.state(), o.chain_state()
        check_invariants(s, cfg, prev, ctx=f"t={t}")
        prev = s
        dropped = s["rej_nomodel"].sum() + s["rej_overflow"].sum()
        in_flight = s["qlen"].sum() + s["busy"].sum() + ch["pending_count"].sum()
        assert queries == ch["q_done"].sum() + dropped + in_flight, t
        for e in range(cfg["E"]):
            for m in range(cfg["M"]):
                n = int(s["qlen"][e, m])
                qc, qe = ch["queue_chain"][e, m, :n], s["queues"][e, m, :n]
                assert np.all(qc[:, 1] < qc[:, 2])                       # k < n_steps
                assert np.all(qc[:, 5] - qe[:, 4] >= qc[:, 1])            # beta - budget >= k
                busy = s["slots"][e, m][:, 0] >= 0
                sc, se = ch["slot_chain"][e, m][busy], s["slots"][e, m][busy]
                assert np.all(sc[:, 5] - se[:, 3] >= sc[:, 1])
            pc = int(ch["pending_count"][e])
            p = ch["pending"][e, :pc]
            assert np.all((p[:, 1] >= 1) & (p[:, 1] < p[:, 2]))
            assert np.all(p[:, 6] - p[:, 5] <= t + 1 - p[:, 1])           # t_arrive <= t + 1 - k
    assert ch["q_done"].sum() > 50 and ch["pending_count"].sum() > 0


def test_bad_n_steps_env_untouched():
    cfg = workload.configs.get("c2c", E=3, T=10)
    o, _ = make_oracle(cfg, seed=6, Q=64)
    cnt = workload.gen.counts(cfg, 6)
    for t in range(6):
        o.tick(workload.gen.tick(cfg, 6, t, cnt[t], 64))
    arr = workload.gen.tick(cfg, 6, 6, np.array([2, 3, 2], np.int32), 64)
    arr["n_steps"] = arr["n_steps"].copy()
    arr["n_steps"][2] = cfg["max_steps"] + 1      # env 1
    before, ch0 = o.state(), o.chain_state()
    o.tick(arr)
    assert o.error & oracle.ERR_STEPS
    after, ch1 = o.state(), o.chain_state()
    for k in ("qlen", "enqueued", "started", "completed"):
        np.testing.assert_array_equal(after[k][1], before[k][1], err_msg=k)
    assert ch1["pending_count"][1] == ch0["pending_count"][1]
    np.testing.assert_array_equal(ch1["pending"][1], ch0["pending"][1])
    arr["n_steps"][2] = 0
    o.clear_error()
    o.tick(arr)
    assert o.error & oracle.ERR_STEPS


def test_dual_pool_rotates_roles():
    cfg = workload.configs.get("c2d", E=2, T=12, embed_dim=64, max_steps=4, lam=6.0)
    o, (P, roles, emb, cap, lb) = make_oracle(cfg, seed=7, Q=64)
    cnt = workload.gen.counts(cfg, 7)
    checked = 0
    for t in range(10):
        arr = workload.gen.tick(cfg, 7, t, cnt[t], 64)
        ch = o.chain_state()
        ro = o.row_offsets(arr)
        act, lg = o.route(arr)
        for e in range(cfg["E"]):
            for i in range(int(ch["pending_count"][e])):
                q_idx, k, n, role0, base, beta, dl = ch["pending"][e, i]
                z = o.dual_trace(e, int(q_idx), int((role0 + k) % cfg["n_roles"]), int(dl) - t)["z"]
                np.testing.assert_array_equal(lg[ro[e] + i], z[:cfg["A"]])
                checked += 1
        o.schedule(arr, act)
    assert checked > 5


def test_broken_csr_skips_every_env():
    """Chain pools lay each env's rows out by a scan over the arrival offsets,
    so offsets that are not one monotone partition of [0, n_total) (here env 2
    re-reads env 0's records) make no arrival usable: every env keeps its
    state and pending calls, only the tick advances; a single-step pool with
    the same offsets still judges each env on its own range."""
    cfg = workload.configs.get("c2c", E=3, T=10)
    o, _ = make_oracle(cfg, seed=8, Q=64)
    cnt = workload.gen.counts(cfg, 8)
    for t in range(6):
        o.tick(workload.gen.tick(cfg, 8, t, cnt[t], 64))
    arr = workload.gen.tick(cfg, 8, 6, np.array([4, 2, 2], np.int32), 64)
    arr["offsets"] = np.array([0, 4, 2, 8], np.int32)     # env 1 [4, 2), env 2 [2, 8)
    before, ch0, t0 = o.state(), o.chain_state(), o.t
    ro = o.row_offsets(arr)
    np.testing.assert_array_equal(np.diff(ro), ch0["pending_count"])   # pending calls only
    o.tick(arr)
    assert o.error & oracle.ERR_COUNT and o.t == t0 + 1
    after, ch1 = o.state(), o.chain_state()
    for k in ("qlen", "enqueued", "started", "completed", "arrived", "busy", "ewma", "backlog"):
        np.testing.assert_array_equal(after[k], before[k], err_msg=k)
    np.testing.assert_array_equal(ch1["pending_count"], ch0["pending_count"])
    np.testing.assert_array_equal(ch1["pending"], ch0["pending"])
    # single-step pool: env 1 alone is rejected, envs 0 and 2 are served
    cfg1 = workload.configs.get("c2", E=3, T=10)
    o1, _ = make_oracle(cfg1, seed=8, Q=64)
    arr1 = {k: v for k, v in arr.items() if k != "n_steps"}
    o1.tick(arr1)
    assert o1.error & oracle.ERR_COUNT
    s1 = o1.state()
    assert s1["arrived"][0] == 4 and s1["arrived"][1] == 0 and s1["arrived"][2] == 6
