"""ctypes binding of libinframind (include/inframind.h): argument marshalling
only. Every step of the tick runs in the library's HIP kernels; torch tensors
merely provide device memory and the current HIP stream.

The functions keep the C names (im_pool_create, im_pool_create_dual, im_route, im_route_sample,
im_schedule, im_tick, im_destroy, im_read_state, im_write_state,
im_set_enabled, im_set_capacity, im_get_error, im_clear_error, im_last_error)."""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libinframind.so")

IM_OK, IM_EINVAL, IM_ENOMEM, IM_EHIP, IM_EDEVICE, IM_ESTATE, IM_EUNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
IM_F32, IM_BF16 = 0, 1
KEY_MODES = {"slack": 0, "deadline": 1, "fcfs": 2}
IM_ERR_QIDX, IM_ERR_COUNT, IM_ERR_BUDGET, IM_ERR_SVC, IM_ERR_ACTION, IM_ERR_ROLE = 1, 2, 4, 8, 16, 32
IM_ERR_STEPS = 64
IM_NET_MLP, IM_NET_DUAL = 0, 1

EXPORTED = ("im_pool_create", "im_pool_create_dual", "im_route", "im_route_sample", "im_schedule", "im_tick", "im_destroy",
            "im_dual_update", "im_set_rpm_limit", "im_get_rows", "im_read_chain_state",
            "im_read_state", "im_write_state", "im_write_chain_state", "im_set_enabled", "im_set_capacity",
            "im_get_error", "im_clear_error", "im_last_error", "im_set_launch", "im_tick_noalloc")


class ImPoolDesc(ctypes.Structure):
    _fields_ = [("n_envs", ctypes.c_int32), ("n_models", ctypes.c_int32),
                ("n_depths", ctypes.c_int32), ("queue_cap", ctypes.c_int32),
                ("max_slots", ctypes.c_int32), ("embed_dim", ctypes.c_int32),
                ("feat_dim", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("widths", ctypes.c_int32 * 4), ("dtype", ctypes.c_int32),
                ("key_mode", ctypes.c_int32), ("max_arrivals_per_env_tick", ctypes.c_int32),
                ("budget_max", ctypes.c_int32), ("value_head", ctypes.c_int32),
                ("net", ctypes.c_int32), ("n_roles", ctypes.c_int32),
                ("max_steps", ctypes.c_int32)]


class ImArrivals(ctypes.Structure):
    _fields_ = [("offsets", ctypes.c_void_p), ("q_idx", ctypes.c_void_p),
                ("budget", ctypes.c_void_p), ("base_svc", ctypes.c_void_p),
                ("role", ctypes.c_void_p), ("n_steps", ctypes.c_void_p),
                ("n_total", ctypes.c_int32)]


class ImRows(ctypes.Structure):
    _fields_ = [("offsets", ctypes.c_void_p), ("n_rows", ctypes.c_void_p),
                ("q_idx", ctypes.c_void_p), ("budget", ctypes.c_void_p), ("role", ctypes.c_void_p)]


# im_dual_net fields, in order, and the workload parameter names they take.
DUAL_FIELDS = (("W_sem", "W_sem"), ("b_sem", "b_sem"), ("ln_sem_gain", "g_sem"),
               ("ln_sem_bias", "be_sem"), ("W_bud", "W_bud"), ("b_bud", "b_bud"),
               ("W_sys", "W_sys"), ("b_sys", "b_sys"), ("W_res", "W_res"), ("b_res", "b_res"),
               ("ln_res_gain", "g_res"), ("ln_res_bias", "be_res"), ("W_merge", "W_merge"),
               ("b_merge", "b_merge"), ("W_act", "W_act"), ("b_act", "b_act"))


class ImDualNet(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f, _ in DUAL_FIELDS] + [("role_emb", ctypes.c_void_p)]


class ImPolicyOut(ctypes.Structure):
    _fields_ = [("actions", ctypes.c_void_p), ("logp", ctypes.c_void_p),
                ("entropy", ctypes.c_void_p), ("value", ctypes.c_void_p),
                ("logits", ctypes.c_void_p)]


ENTRY_DT = np.dtype([("key", "<i4"), ("id", "<i4"), ("t_arr", "<i4"), ("svc", "<u2"),
                     ("budget", "<i2")])
CHAIN_DT = np.dtype([("q_idx", "<i4"), ("k", "<i2"), ("n_steps", "<i2"), ("role0", "<i2"),
                     ("base_svc", "<i2"), ("beta", "<i4")])
PENDING_DT = np.dtype([("ch", CHAIN_DT), ("deadline", "<i4")])
SLOT_DT = np.dtype([("id", "<i4"), ("t_arr", "<i4"), ("rem", "<i4"), ("budget", "<i4")])
MODEL_DT = np.dtype([("qlen", "<i4"), ("busy", "<i4"), ("ewma_q8", "<i4"), ("backlog", "<i4"),
                     ("capacity", "<i4"), ("enabled", "<i4"), ("_p0", "<i4"), ("_p1", "<i4"),
                     ("rej_overflow", "<i8"), ("enqueued", "<i8"), ("started", "<i8"),
                     ("completed", "<i8"), ("slo_met", "<i8"), ("lat_sum", "<i8"),
                     ("wait_sum", "<i8"), ("cost_q16", "<i8"), ("rpm_limit", "<i4"),
                     ("rpm_count", "<i4"), ("rpm_hist", "u1", (60,)), ("_p3", "<i4")])
ENV_DT = np.dtype([("arrived", "<i8"), ("rej_nomodel", "<i8"), ("next_id", "<i4"), ("_p", "<i4"),
                   ("q_done", "<i8"), ("q_met", "<i8")])
assert ENTRY_DT.itemsize == 16 and SLOT_DT.itemsize == 16
assert MODEL_DT.itemsize == 168 and ENV_DT.itemsize == 40
assert CHAIN_DT.itemsize == 16 and PENDING_DT.itemsize == 20

_lib = None


def load() -> ctypes.CDLL:
    """Load the in-tree libinframind.so; fails loudly when it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(hipcc, gfx950); there is no fallback path")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.im_pool_create.argtypes = [ctypes.POINTER(ImPoolDesc), P, P, P, I64, P, P, P,
                                 ctypes.POINTER(P)]
    L.im_pool_create_dual.argtypes = [ctypes.POINTER(ImPoolDesc), ctypes.POINTER(ImDualNet), P, I64,
                                      P, P, P, ctypes.POINTER(P)]
    L.im_route.argtypes = [P, ctypes.POINTER(ImArrivals), P, P, P]
    L.im_route_sample.argtypes = [P, ctypes.POINTER(ImArrivals), ctypes.c_uint64, I32,
                                  ctypes.POINTER(ImPolicyOut), P]
    L.im_schedule.argtypes = [P, ctypes.POINTER(ImArrivals), P, P]
    L.im_tick.argtypes = [P, ctypes.POINTER(ImArrivals), P, P]
    L.im_destroy.argtypes = [P]
    L.im_dual_update.argtypes = [P, ctypes.c_double, ctypes.c_double, P, P]
    L.im_destroy.restype = None
    L.im_read_state.argtypes = [P, I32, I32, ctypes.POINTER(I32), P, P, P, P, P]
    L.im_write_state.argtypes = [P, I32, I32, I32, P, P, P, P, P]
    L.im_write_chain_state.argtypes = [P, I32, I32, I32, P, P, P, P, P, P, P, P, P]
    L.im_set_enabled.argtypes = [P, I32, I32, I32, P]
    L.im_set_capacity.argtypes = [P, I32, I32, I32, P]
    L.im_set_rpm_limit.argtypes = [P, I32, I32, I32, P]
    L.im_set_launch.argtypes = [P, I32, I32]
    L.im_tick_noalloc.argtypes = [P, ctypes.POINTER(ImArrivals), P]
    L.im_get_rows.argtypes = [P, ctypes.POINTER(ImRows)]
    L.im_read_chain_state.argtypes = [P, I32, I32, P, P, P, P]
    L.im_get_error.argtypes = [P, ctypes.POINTER(I32)]
    L.im_clear_error.argtypes = [P]
    L.im_last_error.argtypes = [P]
    L.im_last_error.restype = ctypes.c_char_p
    for name in EXPORTED:
        if name not in ("im_destroy", "im_last_error"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


class IMError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def _check(status, pool=None):
    if status != IM_OK:
        raise IMError(status, load().im_last_error(pool).decode())
    return status


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _hptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def make_desc(cfg: dict) -> ImPoolDesc:
    d = ImPoolDesc()
    d.n_envs, d.n_models, d.n_depths = cfg["E"], cfg["M"], cfg["K"]
    d.queue_cap, d.max_slots = cfg["qcap"], cfg["max_slots"]
    d.embed_dim, d.feat_dim = cfg["embed_dim"], cfg["feat_dim"]
    d.dtype = IM_BF16 if cfg["dtype"] == "bf16" else IM_F32
    d.key_mode = KEY_MODES[cfg["key_mode"]]
    d.max_arrivals_per_env_tick = cfg["max_arrivals"]
    d.budget_max = cfg["budget_max"]
    vh = 1 if cfg.get("value_head") else 0
    d.value_head = vh
    d.max_steps = int(cfg.get("max_steps", 1))
    if cfg.get("net") == "dual":
        d.net, d.n_roles = IM_NET_DUAL, cfg["n_roles"]
        return d
    d.n_layers = len(cfg["widths"])
    for i, w in enumerate(cfg["widths"]):
        d.widths[i] = w
    d.widths[d.n_layers - 1] = cfg["widths"][-1] + vh
    return d


def make_arrivals(offsets, q_idx, budget, base_svc, role=None, n_steps=None) -> ImArrivals:
    """Arrivals of one tick from device tensors (int32, int32, int16, int16;
    int16 roles for dual-pathway pools, int16 calls per query for chain pools)."""
    a = ImArrivals()
    a.offsets = offsets.data_ptr()
    a.q_idx = q_idx.data_ptr() if q_idx.numel() else None
    a.budget = budget.data_ptr() if budget.numel() else None
    a.base_svc = base_svc.data_ptr() if base_svc.numel() else None
    a.role = role.data_ptr() if role is not None and role.numel() else None
    a.n_steps = n_steps.data_ptr() if n_steps is not None and n_steps.numel() else None
    a.n_total = int(q_idx.numel())
    a._keep = (offsets, q_idx, budget, base_svc, role, n_steps)
    return a


def im_pool_create(desc: ImPoolDesc, W, b, emb, n_queries: int, capacity, logit_bias=None,
                   stream=None) -> ctypes.c_void_p:
    """W, b: lists of host float32 arrays; emb: device tensor (borrowed: the
    caller keeps it alive); capacity: host int32 [E*M]."""
    L = load()
    Wc = [np.ascontiguousarray(w, np.float32) for w in W]
    bc = [np.ascontiguousarray(x, np.float32) for x in b]
    Wp = (ctypes.c_void_p * len(Wc))(*[w.ctypes.data for w in Wc])
    bp = (ctypes.c_void_p * len(bc))(*[x.ctypes.data for x in bc])
    cap = np.ascontiguousarray(capacity, np.int32).reshape(-1)
    lb = None if logit_bias is None else np.ascontiguousarray(logit_bias, np.float32)
    out = ctypes.c_void_p()
    _check(L.im_pool_create(ctypes.byref(desc), ctypes.cast(Wp, ctypes.c_void_p),
                            ctypes.cast(bp, ctypes.c_void_p), _dptr(emb), int(n_queries),
                            _hptr(cap), None if lb is None else _hptr(lb), _stream(stream),
                            ctypes.byref(out)))
    return out


def im_pool_create_dual(desc: ImPoolDesc, params: dict, roles, emb, n_queries: int, capacity,
                        logit_bias=None, stream=None) -> ctypes.c_void_p:
    """params: host float32 arrays of the dual-pathway executor (names of
    workload.gen.dual_weights); roles: host float32 [n_roles, E_d]; emb: device
    tensor (borrowed); capacity: host int32 [E*M]."""
    L = load()
    keep = {f: np.ascontiguousarray(params[k], np.float32) for f, k in DUAL_FIELDS}
    keep["role_emb"] = np.ascontiguousarray(roles, np.float32)
    net = ImDualNet(**{f: v.ctypes.data for f, v in keep.items()})
    cap = np.ascontiguousarray(capacity, np.int32).reshape(-1)
    lb = None if logit_bias is None else np.ascontiguousarray(logit_bias, np.float32)
    out = ctypes.c_void_p()
    _check(L.im_pool_create_dual(ctypes.byref(desc), ctypes.byref(net), _dptr(emb), int(n_queries),
                                 _hptr(cap), None if lb is None else _hptr(lb), _stream(stream),
                                 ctypes.byref(out)))
    return out


def im_route(pool, arr: ImArrivals, actions, logits=None, stream=None):
    _check(load().im_route(pool, ctypes.byref(arr), _dptr(actions), _dptr(logits),
                           _stream(stream)), pool)


def im_route_sample(pool, arr: ImArrivals, seed: int, greedy: bool, actions, logp=None,
                    entropy=None, value=None, logits=None, stream=None):
    """RL-rollout route: device tensors for the outputs (None to skip)."""
    out = ImPolicyOut(_dptr(actions), _dptr(logp), _dptr(entropy), _dptr(value), _dptr(logits))
    _check(load().im_route_sample(pool, ctypes.byref(arr), int(seed) & 0xffffffffffffffff,
                                  int(bool(greedy)), ctypes.byref(out), _stream(stream)), pool)


def im_schedule(pool, arr: ImArrivals, actions, stream=None):
    _check(load().im_schedule(pool, ctypes.byref(arr), _dptr(actions), _stream(stream)), pool)


def im_tick(pool, arr: ImArrivals, actions_out=None, stream=None):
    _check(load().im_tick(pool, ctypes.byref(arr), _dptr(actions_out), _stream(stream)), pool)


def im_tick_noalloc(pool, arr: ImArrivals, stream=None):
    """im_tick with the actions staged in the library's static device array."""
    _check(load().im_tick_noalloc(pool, ctypes.byref(arr), _stream(stream)), pool)


def im_dual_update(pool, eta: float, lambda_max: float, lam, stream=None):
    """Eq. 7 on the device; `lam` is a device float64 tensor [1] (in/out)."""
    _check(load().im_dual_update(pool, float(eta), float(lambda_max), _dptr(lam), _stream(stream)), pool)


_hip = None


def device_to_host(ptr, dtype, count) -> np.ndarray:
    """Copy `count` elements of `dtype` from a device pointer the library
    returned (hipMemcpy of the HIP runtime; synchronises)."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipDeviceSynchronize.restype = ctypes.c_int
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    out = np.empty(count, dtype)
    if count:
        if _hip.hipDeviceSynchronize() != 0 or _hip.hipMemcpy(_hptr(out), ptr, out.nbytes, 2) != 0:
            raise RuntimeError("hipMemcpy device-to-host failed")
    return out


def im_get_rows(pool) -> ImRows:
    """Chain pools: device pointers to the current tick's rows."""
    r = ImRows()
    _check(load().im_get_rows(pool, ctypes.byref(r)), pool)
    return r


def im_read_chain_state(pool, env_begin: int, env_count: int, M: int, S: int, qcap: int) -> dict:
    """Chain pools: chain words of the queued calls (service order, like
    im_read_state's queues) and of the busy slots, the pending calls and their
    counts, as numpy arrays in the oracle's chain_state layout (without the
    query counters, which im_read_state reports per env)."""
    E = env_count
    q = np.zeros(E * M * qcap, CHAIN_DT)
    sl = np.zeros(E * M * S, CHAIN_DT)
    pend = np.zeros(E * M * S, PENDING_DT)
    pc = np.zeros(E, np.int32)
    _check(load().im_read_chain_state(pool, env_begin, env_count, _hptr(q), _hptr(sl), _hptr(pend),
                                      _hptr(pc)), pool)

    def six(c):
        return np.stack([c["q_idx"], c["k"], c["n_steps"], c["role0"], c["base_svc"], c["beta"]],
                        axis=-1).astype(np.int32)
    pe = np.concatenate([six(pend["ch"]), pend["deadline"][:, None].astype(np.int32)], axis=-1)
    return dict(queue_chain=six(q).reshape(E, M, qcap, 6), slot_chain=six(sl).reshape(E, M, S, 6),
                pending=pe.reshape(E, M * S, 7), pending_count=pc)


def im_destroy(pool):
    if pool:
        load().im_destroy(pool)


def im_set_enabled(pool, env, model, enabled, stream=None):
    _check(load().im_set_enabled(pool, env, model, int(bool(enabled)), _stream(stream)), pool)


def im_set_capacity(pool, env, model, capacity, stream=None):
    _check(load().im_set_capacity(pool, env, model, int(capacity), _stream(stream)), pool)


def im_set_rpm_limit(pool, env, model, rpm_limit, stream=None):
    _check(load().im_set_rpm_limit(pool, env, model, int(rpm_limit), _stream(stream)), pool)


def im_set_launch(pool, route_blocks: int, sched_waves: int = 0):
    _check(load().im_set_launch(pool, int(route_blocks), int(sched_waves)), pool)


def im_get_error(pool) -> int:
    bits = ctypes.c_int32(0)
    st = load().im_get_error(pool, ctypes.byref(bits))
    if st not in (IM_OK, IM_EDEVICE):
        _check(st, pool)
    return int(bits.value)


def im_clear_error(pool):
    _check(load().im_clear_error(pool), pool)


def im_last_error(pool=None) -> str:
    return load().im_last_error(pool).decode()


def im_read_state(pool, env_begin: int, env_count: int, M: int, A: int, S: int, qcap: int,
                  with_queues: bool = True) -> dict:
    """Snapshot of envs [env_begin, env_begin + env_count) as numpy arrays in
    the layout the tests compare (same keys as the oracle's snapshot).
    with_queues=False skips the queue contents (then "queues" is None)."""
    E = env_count
    envs = np.zeros(E, ENV_DT)
    models = np.zeros(E * M, MODEL_DT)
    slots = np.zeros(E * M * S, SLOT_DT)
    queues = np.zeros(E * M * (qcap if with_queues else 1), ENTRY_DT)
    hist = np.zeros(E * A, np.int64)
    tick = ctypes.c_int32(0)
    _check(load().im_read_state(pool, env_begin, env_count, ctypes.byref(tick), _hptr(envs),
                                _hptr(models), _hptr(slots),
                                _hptr(queues) if with_queues else None, _hptr(hist)), pool)
    md = models.reshape(E, M)
    qarr = None
    if with_queues:
        q = queues.reshape(E, M, qcap)
        qarr = np.stack([q["key"], q["id"], q["t_arr"], q["svc"].astype(np.int32),
                         q["budget"].astype(np.int32)], axis=-1).astype(np.int32)
    sl = slots.reshape(E, M, S)
    sarr = np.stack([sl["id"], sl["t_arr"], sl["rem"], sl["budget"]], axis=-1).astype(np.int32)
    out = dict(t=int(tick.value), next_id=envs["next_id"].copy(), arrived=envs["arrived"].copy(),
               rej_nomodel=envs["rej_nomodel"].copy(), slots=sarr, queues=qarr,
               hist=hist.reshape(E, A), q_done=envs["q_done"].copy(), q_met=envs["q_met"].copy())
    for k, f in (("qlen", "qlen"), ("busy", "busy"), ("ewma", "ewma_q8"), ("backlog", "backlog"),
                 ("cap", "capacity"), ("enabled", "enabled"), ("rej_overflow", "rej_overflow"),
                 ("enqueued", "enqueued"), ("started", "started"), ("completed", "completed"),
                 ("slo_met", "slo_met"), ("lat_sum", "lat_sum"), ("wait_sum", "wait_sum"),
                 ("cost_q16", "cost_q16"), ("rpm_limit", "rpm_limit"), ("rpm_count", "rpm_count")):
        out[k] = md[f].astype(np.int64)
    out["rpm_hist"] = md["rpm_hist"].copy()
    return out


def _state_arrays(s: dict):
    """Host arrays of a state dict in im_read_state's layout."""
    E, M = s["qlen"].shape
    A = s["hist"].shape[1]
    S = s["slots"].shape[2]
    qcap = s["queues"].shape[2]
    envs = np.zeros(E, ENV_DT)
    envs["arrived"], envs["rej_nomodel"], envs["next_id"] = s["arrived"], s["rej_nomodel"], s["next_id"]
    if "q_done" in s:
        envs["q_done"], envs["q_met"] = s["q_done"], s["q_met"]
    models = np.zeros((E, M), MODEL_DT)
    for k, f in (("qlen", "qlen"), ("busy", "busy"), ("ewma", "ewma_q8"), ("backlog", "backlog"),
                 ("cap", "capacity"), ("enabled", "enabled"), ("rej_overflow", "rej_overflow"),
                 ("enqueued", "enqueued"), ("started", "started"), ("completed", "completed"),
                 ("slo_met", "slo_met"), ("lat_sum", "lat_sum"), ("wait_sum", "wait_sum"),
                 ("cost_q16", "cost_q16"), ("rpm_limit", "rpm_limit"), ("rpm_count", "rpm_count")):
        models[f] = s[k]
    models["rpm_hist"] = s["rpm_hist"]
    slots = np.zeros((E, M, S), SLOT_DT)
    for i, f in enumerate(("id", "t_arr", "rem", "budget")):
        slots[f] = s["slots"][..., i]
    queues = np.zeros((E, M, qcap), ENTRY_DT)
    for i, f in enumerate(("key", "id", "t_arr", "svc", "budget")):
        queues[f] = s["queues"][..., i]
    hist = np.ascontiguousarray(s["hist"], np.int64)
    return E, envs, models, slots, queues, hist


def im_write_state(pool, env_begin: int, s: dict):
    """Inverse of im_read_state (same dict layout)."""
    E, envs, models, slots, queues, hist = _state_arrays(s)
    _check(load().im_write_state(pool, env_begin, E, int(s["t"]), _hptr(envs), _hptr(models),
                                 _hptr(slots), _hptr(queues), _hptr(hist)), pool)


def im_write_chain_state(pool, env_begin: int, s: dict, c: dict):
    """Restore a chain pool: s as from im_read_state, c as from
    im_read_chain_state (queue_chain, slot_chain, pending, pending_count)."""
    E, envs, models, slots, queues, hist = _state_arrays(s)

    def chains(six):
        out = np.zeros(six.shape[:-1], CHAIN_DT)
        for i, f in enumerate(("q_idx", "k", "n_steps", "role0", "base_svc", "beta")):
            out[f] = six[..., i]
        return out
    qch = chains(np.asarray(c["queue_chain"]))
    sch = chains(np.asarray(c["slot_chain"]))
    pe = np.asarray(c["pending"])
    pend = np.zeros(pe.shape[:-1], PENDING_DT)
    pend["ch"] = chains(pe[..., :6])
    pend["deadline"] = pe[..., 6]
    pc = np.ascontiguousarray(c["pending_count"], np.int32)
    _check(load().im_write_chain_state(pool, env_begin, E, int(s["t"]), _hptr(envs), _hptr(models),
                                       _hptr(slots), _hptr(queues), _hptr(hist), _hptr(qch), _hptr(sch),
                                       _hptr(pend), _hptr(pc)), pool)
