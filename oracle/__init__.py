"""ctypes front end of the CPU oracle of the route-and-schedule tick.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark may use it; the GPU library never does. The oracle is plain
scalar C++ (oracle.cpp) with the policy MLP in fp64; see that file for the
paper passages each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
# IM_ORACLE_LIB: another build of oracle.cpp (the sanitizer test loads one
# built with AddressSanitizer and UBSan)
_LIB = os.environ.get("IM_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

KEY_MODES = {"slack": 0, "deadline": 1, "fcfs": 2}
ERR_QIDX, ERR_COUNT, ERR_BUDGET, ERR_SVC, ERR_ACTION, ERR_ROLE, ERR_STEPS = 1, 2, 4, 8, 16, 32, 64

# Parameters of the dual-pathway executor, in the order orc_create_dual takes them.
DUAL_PARAMS = ("W_sem", "b_sem", "g_sem", "be_sem", "W_bud", "b_bud", "W_sys", "b_sys",
               "W_res", "b_res", "g_res", "be_res", "W_merge", "b_merge", "W_act", "b_act")


def build(force: bool = True) -> str:
    """Compile oracle.cpp into liboracle.so with g++ (no GPU involved)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread",
                               "-ffp-contract=off", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Desc(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int32), ("M", ctypes.c_int32), ("K", ctypes.c_int32),
                ("qcap", ctypes.c_int32), ("max_slots", ctypes.c_int32),
                ("embed_dim", ctypes.c_int32), ("feat_dim", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("widths", ctypes.c_int32 * 4),
                ("dtype", ctypes.c_int32), ("key_mode", ctypes.c_int32),
                ("max_arrivals", ctypes.c_int32), ("budget_max", ctypes.c_int32),
                ("value_head", ctypes.c_int32), ("net", ctypes.c_int32),
                ("n_roles", ctypes.c_int32), ("max_steps", ctypes.c_int32), ("Q", ctypes.c_int64)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        L.orc_create.restype = P
        L.orc_create.argtypes = [ctypes.POINTER(_Desc), P, P, P, P, P]
        L.orc_destroy.argtypes = [P]
        L.orc_tick.argtypes = [P]
        L.orc_tick.restype = ctypes.c_int32
        L.orc_error.argtypes = [P]
        L.orc_error.restype = ctypes.c_int32
        L.orc_clear_error.argtypes = [P]
        L.orc_create_dual.restype = P
        L.orc_create_dual.argtypes = [ctypes.POINTER(_Desc), P, P, P, P, P]
        L.orc_dual_trace.argtypes = [P, ctypes.c_int, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P]
        I32 = ctypes.c_int32
        L.orc_route.argtypes = [P, I32, P, P, P, P, P, P, P, ctypes.c_int]
        L.orc_schedule.argtypes = [P, I32, P, P, P, P, P, P, P, ctypes.c_int]
        L.orc_row_offsets.argtypes = [P, I32, P, P]
        L.orc_read_chain.argtypes = [P, P, P, P, P, P]
        L.orc_features.argtypes = [P, ctypes.c_int, ctypes.c_int32, ctypes.c_int32, P]
        L.orc_round_bf16.argtypes = [ctypes.c_double]
        L.orc_round_bf16.restype = ctypes.c_double
        L.orc_round_bf16_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        L.orc_set_enabled.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.orc_set_capacity.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.orc_read_state.argtypes = [P] * 7
        U32 = ctypes.c_uint32
        L.orc_route_rl.argtypes = [P, ctypes.c_int, I32, P, P, P, P, P, U32, U32, ctypes.c_int, P,
                                   P, P, P, P, ctypes.c_int]
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_gumbel.argtypes = [U32, U32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int]
        L.orc_gumbel.restype = ctypes.c_double
        L.orc_dual_update.argtypes = [P, ctypes.c_double, ctypes.c_double, P]
        L.orc_set_rpm_limit.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.orc_read_rpm.argtypes = [P, P, P, P]
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def philox4x32_10(ctr, key) -> np.ndarray:
    """One Philox4x32-10 block: uint32 [4] from counter uint32 [4], key uint32 [2]."""
    c = np.ascontiguousarray(ctr, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.empty(4, np.uint32)
    _load().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def gumbel(seed: int, req_id: int, env: int, action: int) -> float:
    """Gumbel noise the sampler adds to the logit of `action` of request
    `req_id` of env `env` (global env index) under `seed`."""
    return _load().orc_gumbel(seed & 0xffffffff, (seed >> 32) & 0xffffffff, req_id, env, action)


def round_bf16(v: float) -> float:
    return _load().orc_round_bf16(float(v))


def round_bf16_array(x) -> np.ndarray:
    """bf16 round-to-nearest-even of every element (fp64 in, fp64 out)."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty_like(x)
    _load().orc_round_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


class Oracle:
    """One oracle pool over E envs (cfg: a workload config dict).

    W, b: lists of fp32 arrays (W[l] is [out, in]); emb_values: float32
    [Q, E_d] (the value of each table entry); cap: int32 [E, M];
    logit_bias: float32 [M] or None. For a dual-pathway executor
    (cfg["net"] == "dual", Sec. 4.2) W is a dict of its fp32 parameters
    (names in DUAL_PARAMS), b is unused and roles is the fp32 role-embedding
    table [n_roles, E_d]."""

    def __init__(self, cfg, W, b, emb_values, cap, logit_bias=None, E=None, threads=1, roles=None):
        L = _load()
        d = _Desc()
        self.E = cfg["E"] if E is None else E
        self.dual = cfg.get("net") == "dual"
        d.E, d.M, d.K = self.E, cfg["M"], cfg["K"]
        d.qcap, d.max_slots = cfg["qcap"], cfg["max_slots"]
        vh = 1 if cfg.get("value_head") else 0
        d.value_head = vh
        if self.dual:
            d.embed_dim, d.feat_dim, d.n_layers = cfg["embed_dim"], cfg["embed_dim"] + 4 * cfg["M"] + 1, 0
            d.net, d.n_roles = 1, cfg["n_roles"]
        else:
            d.embed_dim, d.feat_dim, d.n_layers = cfg["embed_dim"], cfg["feat_dim"], len(cfg["widths"])
            for i, w in enumerate(cfg["widths"]):
                d.widths[i] = w
            d.widths[len(cfg["widths"]) - 1] = cfg["widths"][-1] + vh
        d.dtype = 1 if cfg["dtype"] == "bf16" else 0
        d.max_steps = int(cfg.get("max_steps", 1))
        self.chains = d.max_steps > 1
        d.key_mode = KEY_MODES[cfg["key_mode"]]
        d.max_arrivals = cfg["max_arrivals"]
        d.budget_max = cfg["budget_max"]
        emb = np.ascontiguousarray(emb_values, np.float32)
        d.Q = emb.shape[0]
        self.cfg, self.M, self.K, self.A = cfg, cfg["M"], cfg["K"], cfg["M"] * cfg["K"]
        self.qcap, self.S = cfg["qcap"], cfg["max_slots"]
        self.threads = threads
        cap = np.ascontiguousarray(cap, np.int32).reshape(-1)
        assert cap.size == self.E * self.M
        lb = None if logit_bias is None else np.ascontiguousarray(logit_bias, np.float32)
        self._d = d
        if self.dual:
            self._P = [np.ascontiguousarray(W[k], np.float32).reshape(-1) for k in DUAL_PARAMS]
            self._roles = np.ascontiguousarray(roles, np.float32)
            assert self._roles.shape == (cfg["n_roles"], cfg["embed_dim"])
            Pp = (ctypes.c_void_p * len(self._P))(*[w.ctypes.data for w in self._P])
            self.p = L.orc_create_dual(ctypes.byref(d), ctypes.cast(Pp, ctypes.c_void_p),
                                       _ptr(self._roles), _ptr(emb), _ptr(cap),
                                       None if lb is None else _ptr(lb))
        else:
            self._W = [np.ascontiguousarray(w, np.float32) for w in W]
            self._b = [np.ascontiguousarray(x, np.float32) for x in b]
            Wp = (ctypes.c_void_p * len(W))(*[w.ctypes.data for w in self._W])
            bp = (ctypes.c_void_p * len(b))(*[x.ctypes.data for x in self._b])
            self.p = L.orc_create(ctypes.byref(d), ctypes.cast(Wp, ctypes.c_void_p),
                                  ctypes.cast(bp, ctypes.c_void_p), _ptr(emb), _ptr(cap),
                                  None if lb is None else _ptr(lb))
        self._lib = L

    def __del__(self):
        if getattr(self, "p", None):
            self._lib.orc_destroy(self.p)
            self.p = None

    @property
    def t(self) -> int:
        return self._lib.orc_tick(self.p)

    @property
    def error(self) -> int:
        return self._lib.orc_error(self.p)

    def clear_error(self):
        self._lib.orc_clear_error(self.p)

    @staticmethod
    def _arr(arr):
        return (np.ascontiguousarray(arr["offsets"], np.int32),
                np.ascontiguousarray(arr["q_idx"], np.int32),
                np.ascontiguousarray(arr["budget"], np.int16),
                np.ascontiguousarray(arr["base_svc"], np.int16))

    @staticmethod
    def _role(arr):
        r = arr.get("role")
        return None if r is None else np.ascontiguousarray(r, np.int16)

    @staticmethod
    def _opt16(arr, key):
        r = arr.get(key)
        return None if r is None else _ptr(np.ascontiguousarray(r, np.int16))

    def row_offsets(self, arr) -> np.ndarray:
        """Start of each env's rows in the per-row outputs of the next route /
        schedule call: the arrival offsets for single-step pools; for chain
        pools each env's pending calls, then its arrivals (int32 [E + 1])."""
        off = np.ascontiguousarray(arr["offsets"], np.int32)
        out = np.empty(self.E + 1, np.int32)
        self._lib.orc_row_offsets(self.p, int(np.asarray(arr["q_idx"]).size), _ptr(off), _ptr(out))
        return out

    def route(self, arr, want_logits=True):
        """Returns (actions int32 [rows], logits float64 [rows, A] or None);
        rows as in row_offsets (the arrivals for single-step pools)."""
        off, q, bud, _ = self._arr(arr)
        assert off.size == self.E + 1
        n = max(int(self.row_offsets(arr)[-1]), int(q.size)) if self.chains else int(q.size)
        act = np.full(n, -1, np.int32)
        lg = np.zeros((n, self.A), np.float64) if want_logits else None
        ro = self._role(arr)
        self._lib.orc_route(self.p, int(q.size), _ptr(off), _ptr(q), None if ro is None else _ptr(ro),
                            _ptr(bud), self._opt16(arr, "n_steps"), None if lg is None else _ptr(lg),
                            _ptr(act), self.threads)
        return act, lg

    def route_rl(self, arr, seed: int, greedy: bool = False, env_base: int = 0):
        """RL-rollout route: dict of actions int32 [n], logits, logp, entropy,
        value (float64). `env_base` is the global index of this oracle's env 0
        (the Philox counter uses global env indices)."""
        off, q, bud, _ = self._arr(arr)
        assert off.size == self.E + 1
        n = max(int(self.row_offsets(arr)[-1]), int(q.size)) if self.chains else int(q.size)
        out = dict(actions=np.full(n, -1, np.int32), logits=np.zeros((n, self.A), np.float64),
                   logp=np.zeros(n, np.float64), entropy=np.zeros(n, np.float64),
                   value=np.zeros(n, np.float64))
        ro = self._role(arr)
        self._lib.orc_route_rl(self.p, env_base, int(q.size), _ptr(off), _ptr(q),
                               None if ro is None else _ptr(ro), _ptr(bud), self._opt16(arr, "n_steps"),
                               seed & 0xffffffff, (seed >> 32) & 0xffffffff, int(bool(greedy)),
                               _ptr(out["logits"]), _ptr(out["actions"]), _ptr(out["logp"]),
                               _ptr(out["entropy"]), _ptr(out["value"]), self.threads)
        return out

    def dual_update(self, lam: float, eta: float, lambda_max: float) -> float:
        """Eq. 7 over the completions since the previous call; returns lambda."""
        x = np.array([lam], np.float64)
        self._lib.orc_dual_update(self.p, float(eta), float(lambda_max), _ptr(x))
        return float(x[0])

    def schedule(self, arr, actions):
        off, q, bud, svc = self._arr(arr)
        act = np.ascontiguousarray(actions, np.int32)
        ro = self._role(arr)
        self._lib.orc_schedule(self.p, int(q.size), _ptr(off), _ptr(q),
                               None if ro is None else _ptr(ro), _ptr(bud), _ptr(svc),
                               self._opt16(arr, "n_steps"), _ptr(act), self.threads)

    def tick(self, arr):
        act, _ = self.route(arr, want_logits=False)
        self.schedule(arr, act)
        return act

    def features(self, e, q_idx, budget):
        out = np.empty(self._d.feat_dim, np.float64)
        self._lib.orc_features(self.p, e, q_idx, budget, _ptr(out))
        return out

    def dual_trace(self, e, q_idx, role, budget) -> dict:
        """Hidden vectors of one request of env e through the dual-pathway
        executor: h_sem, h_bud, h_sys, h_res, h and z (logits and value row,
        without the logit bias)."""
        assert self.dual
        sizes = [("h_sem", 128), ("h_bud", 16), ("h_sys", 16), ("h_res", 64), ("h", 128),
                 ("z", self.A + self._d.value_head)]
        out = np.empty(sum(n for _, n in sizes), np.float64)
        self._lib.orc_dual_trace(self.p, e, q_idx, role, budget, _ptr(out))
        res, o = {}, 0
        for k, n in sizes:
            res[k] = out[o:o + n]
            o += n
        return res

    def chain_state(self) -> dict:
        """Chain pools: per queued call (queue order, [E, M, qcap, 6]) and per
        slot ([E, M, S, 6]) the fields (q_idx, k, n_steps, role0, base, beta);
        the pending calls [E, M*S, 7] (+ deadline) and their count [E]; the
        completed and on-time queries per env [E, 2]."""
        E, M, S, Qc = self.E, self.M, self.S, self.qcap
        qch = np.zeros((E, M, Qc, 6), np.int32)
        sch = np.zeros((E, M, S, 6), np.int32)
        pend = np.zeros((E, M * S, 7), np.int32)
        pc = np.zeros(E, np.int32)
        qc = np.zeros((E, 2), np.int64)
        self._lib.orc_read_chain(self.p, _ptr(qch), _ptr(sch), _ptr(pend), _ptr(pc), _ptr(qc))
        return dict(queue_chain=qch, slot_chain=sch, pending=pend, pending_count=pc,
                    q_done=qc[:, 0].copy(), q_met=qc[:, 1].copy())

    def set_enabled(self, e, m, v):
        self._lib.orc_set_enabled(self.p, e, m, int(bool(v)))

    def set_capacity(self, e, m, c):
        self._lib.orc_set_capacity(self.p, e, m, int(c))

    def set_rpm_limit(self, e, m, r):
        self._lib.orc_set_rpm_limit(self.p, e, m, int(r))

    def state(self) -> dict:
        """Snapshot as a dict of numpy arrays (common test representation)."""
        E, M, S, Qc, A = self.E, self.M, self.S, self.qcap, self.A
        env_i32 = np.zeros(E, np.int32)
        env_i64 = np.zeros((E, 2), np.int64)
        mod = np.zeros((E, M, 14), np.int64)
        slots = np.zeros((E, M, S, 4), np.int32)
        queues = np.zeros((E, M, Qc, 5), np.int32)
        hist = np.zeros((E, A), np.int64)
        self._lib.orc_read_state(self.p, _ptr(env_i32), _ptr(env_i64), _ptr(mod), _ptr(slots),
                                 _ptr(queues), _ptr(hist))
        rpm_lim = np.zeros((E, M), np.int32)
        rpm_cnt = np.zeros((E, M), np.int32)
        rpm_hist = np.zeros((E, M, 60), np.uint8)
        self._lib.orc_read_rpm(self.p, _ptr(rpm_lim), _ptr(rpm_cnt), _ptr(rpm_hist))
        return dict(t=self.t, next_id=env_i32, arrived=env_i64[:, 0], rej_nomodel=env_i64[:, 1],
                    qlen=mod[..., 0], busy=mod[..., 1], ewma=mod[..., 2], backlog=mod[..., 3],
                    cap=mod[..., 4], enabled=mod[..., 5], rej_overflow=mod[..., 6],
                    enqueued=mod[..., 7], started=mod[..., 8], completed=mod[..., 9],
                    slo_met=mod[..., 10], lat_sum=mod[..., 11], wait_sum=mod[..., 12],
                    cost_q16=mod[..., 13], rpm_limit=rpm_lim.astype(np.int64),
                    rpm_count=rpm_cnt.astype(np.int64), rpm_hist=rpm_hist,
                    slots=slots, queues=queues, hist=hist)
