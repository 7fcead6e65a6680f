"""Helpers for the GPU parity tests: build a GPU pool and an oracle over a
subset of its envs from the same seeded inputs, and run them in lockstep."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workload
from helpers import assert_state_equal, check_invariants, logits_close, near_tie


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch


def rtol_of(cfg):
    return 2e-2 if cfg["dtype"] == "bf16" else 1e-4


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class Pair:
    """GPU pool over all envs + oracle over envs [e0, e1)."""

    def __init__(self, cfg, seed=0, Q=None, bias_scale=0.1, e0=0, e1=None, threads=8):
        torch = need_gpu()
        import paper_2606_11440_amd as P
        self.cfg, self.seed = cfg, seed
        self.Q = workload.gen.table_rows(cfg) if Q is None else Q
        self.e0, self.e1 = e0, (cfg["E"] if e1 is None else e1)
        W, b = workload.gen.weights(cfg, seed, bias_scale)
        table, emb_vals = workload.gen.embedding(cfg, seed, rows=self.Q)
        cap = workload.gen.capacities(cfg, seed)
        lb = workload.gen.logit_bias(cfg)
        if cfg["dtype"] == "bf16":
            emb_dev = torch.from_numpy(table.view(np.int16)).cuda()
        else:
            emb_dev = torch.from_numpy(table).cuda()
        self.gpu = P.Pool(cfg, W, b, emb_dev, cap, lb)
        self.orc = oracle.Oracle(cfg, W, b, emb_vals, cap[self.e0:self.e1], lb,
                                 E=self.e1 - self.e0, threads=threads)
        self.counts = workload.gen.counts(cfg, seed)
        self.flips = 0
        self.rows_checked = 0
        self.P = P
        self.torch = torch

    def arrivals(self, t):
        return workload.gen.tick(self.cfg, self.seed, t, self.counts[t], self.Q)

    def step(self, arr, mode="route+schedule", check_logits=True):
        """One lockstep tick. mode: 'route+schedule' (im_route with logits,
        then im_schedule) or 'tick' (im_tick with actions_out)."""
        torch, P = self.torch, self.P
        cfg = self.cfg
        dev = P.device_arrivals(arr)
        n = int(arr["q_idx"].size)
        act = torch.full((max(n, 1),), -7, dtype=torch.int32, device="cuda")
        sub = workload.gen.subset(arr, self.e0, self.e1)
        lo = int(arr["offsets"][self.e0])
        ns = int(sub["q_idx"].size)
        if mode == "tick":
            self.gpu.tick(dev, act)
            torch.cuda.synchronize()
            g_act = act[lo:lo + ns].cpu().numpy() if ns else np.zeros(0, np.int32)
            o_act, o_lg = self.orc.route(sub)
            self._check_actions(g_act, o_act, o_lg, None)
        else:
            lg = torch.full((max(n, 1), cfg["A"]), float("nan"), dtype=torch.float32, device="cuda")
            self.gpu.route(dev, act, lg if check_logits else None)
            torch.cuda.synchronize()
            g_act = act[lo:lo + ns].cpu().numpy() if ns else np.zeros(0, np.int32)
            g_lg = lg[lo:lo + ns].cpu().numpy().astype(np.float64) if ns else None
            o_act, o_lg = self.orc.route(sub)
            self._check_actions(g_act, o_act, o_lg, g_lg if check_logits else None)
            self.gpu.schedule(dev, act)
        self.orc.schedule(sub, g_act)
        return g_act

    def _check_actions(self, g_act, o_act, o_lg, g_lg):
        rtol = rtol_of(self.cfg)
        if g_lg is not None and g_act.size:
            ok = logits_close(g_lg, o_lg, rtol)
            if not ok.all():
                r = int(np.argmin(ok))
                raise AssertionError(f"logits outside tolerance at row {r}: gpu {g_lg[r]} "
                                     f"oracle {o_lg[r]}")
        diff = np.nonzero(g_act != o_act)[0]
        for r in diff:
            if not near_tie(o_lg[r], int(o_act[r]), int(g_act[r]), rtol):
                raise AssertionError(f"argmax differs beyond a near tie at row {r}: gpu "
                                     f"{g_act[r]} oracle {o_act[r]} logits {o_lg[r]}")
        self.flips += int(diff.size)
        self.rows_checked += int(g_act.size)

    def compare_state(self, ctx="", invariants=True):
        g = self.gpu.state(self.e0, self.e1 - self.e0)
        o = self.orc.state()
        assert_state_equal(g, o, ctx=ctx)
        if invariants:
            check_invariants(g, self.cfg, ctx=ctx)
        return g

    def close(self):
        self.gpu.close()
