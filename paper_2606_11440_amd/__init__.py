"""MI355X-native batched route-and-schedule tick (InfraMind's executor and
budget-aware queues, vectorised over independent serving pools).

The compute path is libinframind.so (HIP kernels for gfx950 behind the C ABI of
include/inframind.h); this package only marshals arguments. Importing it does
not load the library; the first call does, and fails loudly if it is missing."""
from __future__ import annotations

import numpy as np

from . import _lib
from ._lib import (EXPORTED, IMError, im_clear_error, im_destroy, im_dual_update,  # noqa: F401
                   im_get_error,
                   im_get_rows, im_last_error, im_pool_create, im_pool_create_dual,
                   im_read_chain_state, im_read_state, im_route,
                   im_route_sample,
                   im_schedule,
                   im_set_capacity, im_set_enabled, im_set_launch, im_set_rpm_limit, im_tick,
                   im_tick_noalloc,
                   im_write_chain_state,
                   im_write_state,
                   make_arrivals,
                   make_desc)


def device_arrivals(arr: dict, device="cuda"):
    """Upload one tick's numpy arrivals (offsets, q_idx, budget, base_svc and,
    when present, role)."""
    import torch
    t = lambda x, dt: torch.as_tensor(x, dtype=dt).to(device)  # noqa: E731
    role = t(arr["role"], torch.int16) if "role" in arr else None
    steps = t(arr["n_steps"], torch.int16) if "n_steps" in arr else None
    return make_arrivals(t(arr["offsets"], torch.int32), t(arr["q_idx"], torch.int32),
                         t(arr["budget"], torch.int16), t(arr["base_svc"], torch.int16), role, steps)


class Pool:
    """A pool of E envs on the current GPU, built from a workload config.

    W, b: host float32 weights/biases per layer; emb: device tensor holding the
    embedding table (float32, or bf16 bits as int16/uint16 for bf16 configs),
    kept alive by this object; cap: int32 [E, M]; logit_bias: float32 [M] or None.
    For the dual-pathway executor (cfg["net"] == "dual") W is the parameter
    dict of workload.gen.dual_weights and b the role-embedding table."""

    def __init__(self, cfg, W, b, emb, cap, logit_bias=None, stream=None):
        self.cfg = cfg
        self.E, self.M, self.K = cfg["E"], cfg["M"], cfg["K"]
        self.A, self.S, self.qcap = cfg["M"] * cfg["K"], cfg["max_slots"], cfg["qcap"]
        self.emb = emb
        self.desc = make_desc(cfg)
        if cfg.get("net") == "dual":
            self.h = im_pool_create_dual(self.desc, W, b, emb, emb.shape[0], cap, logit_bias, stream)
        else:
            self.h = im_pool_create(self.desc, W, b, emb, emb.shape[0], cap, logit_bias, stream)

    def route(self, arr, actions, logits=None, stream=None):
        im_route(self.h, arr, actions, logits, stream)

    def route_sample(self, arr, seed, actions, logp=None, entropy=None, value=None, logits=None,
                     greedy=False, stream=None):
        im_route_sample(self.h, arr, seed, greedy, actions, logp, entropy, value, logits, stream)

    def dual_update(self, eta, lambda_max, lam, stream=None):
        im_dual_update(self.h, eta, lambda_max, lam, stream)

    def schedule(self, arr, actions, stream=None):
        im_schedule(self.h, arr, actions, stream)

    def tick(self, arr, actions_out=None, stream=None):
        im_tick(self.h, arr, actions_out, stream)

    def tick_noalloc(self, arr, stream=None):
        im_tick_noalloc(self.h, arr, stream)

    def state(self, env_begin=0, env_count=None, with_queues=True):
        n = self.E - env_begin if env_count is None else env_count
        return im_read_state(self.h, env_begin, n, self.M, self.A, self.S, self.qcap, with_queues)

    def chain_state(self, env_begin=0, env_count=None):
        n = self.E - env_begin if env_count is None else env_count
        return im_read_chain_state(self.h, env_begin, n, self.M, self.S, self.qcap)

    def rows(self):
        """Chain pools: (row offsets int32 [E + 1], row count) of the current
        tick, copied to the host (synchronises)."""
        r = im_get_rows(self.h)
        off = _lib.device_to_host(r.offsets, np.int32, self.E + 1)
        cnt = _lib.device_to_host(r.n_rows, np.int32, 1)
        return off, int(cnt[0])

    def write_state(self, env_begin, s):
        im_write_state(self.h, env_begin, s)

    def write_chain_state(self, env_begin, s, c):
        """Chain pools: s from state(), c from chain_state()."""
        im_write_chain_state(self.h, env_begin, s, c)

    def set_enabled(self, e, m, v, stream=None):
        im_set_enabled(self.h, e, m, v, stream)

    def set_capacity(self, e, m, c, stream=None):
        im_set_capacity(self.h, e, m, c, stream)

    def set_rpm_limit(self, e, m, r, stream=None):
        im_set_rpm_limit(self.h, e, m, r, stream)

    def set_launch(self, route_blocks, sched_waves=0):
        """Launch shapes (results do not depend on them): route_blocks -1
        default, n > 0 persistent grid of n blocks, 0 one wave per tile;
        sched_waves 1, 2 or 4 envs per schedule workgroup (0: keep)."""
        im_set_launch(self.h, route_blocks, sched_waves)

    def error(self) -> int:
        return im_get_error(self.h)

    def clear_error(self):
        im_clear_error(self.h)

    def close(self):
        if getattr(self, "h", None):
            im_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
