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
        if cfg.get("net") == "dual":
            W, b = workload.gen.dual_weights(cfg, seed, bias_scale), workload.gen.roles(cfg, seed)
        else:
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
                                 E=self.e1 - self.e0, threads=threads,
                                 roles=b if cfg.get("net") == "dual" else None)
        self.counts = workload.gen.counts(cfg, seed)
        self.chains = cfg.get("max_steps", 1) > 1
        self.flips = 0
        self.rows_checked = 0
        self.P = P
        self.torch = torch

    def arrivals(self, t):
        return workload.gen.tick(self.cfg, self.seed, t, self.counts[t], self.Q)

    def _rows(self, arr):
        """Capacity of the per-row outputs of a tick (chain pools: the pending
        calls come on top of the arrivals)."""
        n = int(arr["q_idx"].size)
        if self.chains:
            n += self.cfg["E"] * self.cfg["M"] * self.cfg["max_slots"]
        return max(n, 1)

    def _span(self, arr, sub):
        """GPU rows of envs [e0, e1) after a route: (first row, row count)."""
        if self.chains:
            off, _ = self.gpu.rows()
            return int(off[self.e0]), int(off[self.e1] - off[self.e0])
        return int(arr["offsets"][self.e0]), int(sub["q_idx"].size)

    def step(self, arr, mode="route+schedule", check_logits=True):
        """One lockstep tick. mode: 'route+schedule' (im_route with logits,
        then im_schedule) or 'tick' (im_tick with actions_out)."""
        torch, P = self.torch, self.P
        cfg = self.cfg
        dev = P.device_arrivals(arr)
        n = self._rows(arr)
        act = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        sub = workload.gen.subset(arr, self.e0, self.e1)
        if mode == "tick":
            self.gpu.tick(dev, act)
            torch.cuda.synchronize()
            lo, ns = self._span(arr, sub)
            g_act = act[lo:lo + ns].cpu().numpy() if ns else np.zeros(0, np.int32)
            o_act, o_lg = self.orc.route(sub)
            assert o_act.size == ns, (o_act.size, ns)
            self._check_actions(g_act, o_act, o_lg, None)
        else:
            lg = torch.full((n, cfg["A"]), float("nan"), dtype=torch.float32, device="cuda")
            self.gpu.route(dev, act, lg if check_logits else None)
            torch.cuda.synchronize()
            lo, ns = self._span(arr, sub)
            g_act = act[lo:lo + ns].cpu().numpy() if ns else np.zeros(0, np.int32)
            g_lg = lg[lo:lo + ns].cpu().numpy().astype(np.float64) if ns else None
            o_act, o_lg = self.orc.route(sub)
            assert o_act.size == ns, (o_act.size, ns)
            self._check_actions(g_act, o_act, o_lg, g_lg if check_logits else None)
            self.gpu.schedule(dev, act)
        self.orc.schedule(sub, g_act)   # chain pools: the same rows in the same order
        return g_act

    def step_rl(self, arr, seed, greedy=False):
        """One lockstep tick of im_route_sample (sampled or greedy) followed by
        im_schedule with the GPU's actions. Logits, log-probs, entropies and
        values are checked against the oracle within the tolerance; a sampled
        action may differ from the oracle's only where the oracle's perturbed
        scores (logit + its Gumbel noise) of the two are within twice the
        logit tolerance, and the oracle then follows the GPU's action."""
        torch, P = self.torch, self.P
        cfg = self.cfg
        A = cfg["A"]
        vh = bool(cfg.get("value_head"))
        dev = P.device_arrivals(arr)
        nn = self._rows(arr)
        f32 = dict(dtype=torch.float32, device="cuda")
        act = torch.full((nn,), -7, dtype=torch.int32, device="cuda")
        logp = torch.full((nn,), float("nan"), **f32)
        ent = torch.full((nn,), float("nan"), **f32)
        val = torch.full((nn,), float("nan"), **f32) if vh else None
        lg = torch.full((nn, A), float("nan"), **f32)
        self.gpu.route_sample(dev, seed, act, logp, ent, val, lg, greedy=greedy)
        torch.cuda.synchronize()
        sub = workload.gen.subset(arr, self.e0, self.e1)
        lo, ns = self._span(arr, sub)
        sl = slice(lo, lo + ns)
        g_act = act[sl].cpu().numpy()
        g_lg = lg[sl].cpu().numpy().astype(np.float64)
        g_lp = logp[sl].cpu().numpy().astype(np.float64)
        g_en = ent[sl].cpu().numpy().astype(np.float64)
        next_id = self.orc.state()["next_id"]
        o = self.orc.route_rl(sub, seed, greedy=greedy, env_base=self.e0)
        rtol = rtol_of(cfg)
        if ns:
            ok = logits_close(g_lg, o["logits"], rtol)
            if not ok.all():
                r = int(np.argmin(ok))
                raise AssertionError(f"logits outside tolerance at row {r}")
        off = self.orc.row_offsets(sub)
        env_of = np.repeat(np.arange(self.e1 - self.e0), np.diff(off))
        for r in range(ns):
            z = o["logits"][r]
            scale = float(np.max(np.abs(z)))
            ga, oa = int(g_act[r]), int(o["actions"][r])
            lse = z[oa] - o["logp"][r] if oa >= 0 else 0.0
            if ga != oa:
                assert ga >= 0 and oa >= 0, (r, ga, oa)
                e = int(env_of[r])
                rid = int(next_id[e]) + r - int(off[e])
                gn = (lambda a: 0.0) if greedy else (
                    lambda a: oracle.gumbel(seed, rid, self.e0 + e, a))
                margin = (z[oa] + gn(oa)) - (z[ga] + gn(ga))
                assert margin <= 2 * rtol * scale + 1e-5, (r, ga, oa, margin)
                self.flips += 1
            o_lp = z[ga] - lse if ga >= 0 else 0.0
            assert abs(g_lp[r] - o_lp) <= 2 * rtol * scale + 1e-5, ("logp", r, g_lp[r], o_lp)
            tol_h = 2 * np.log(max(A, 2)) * rtol * scale + 1e-5
            assert abs(g_en[r] - o["entropy"][r]) <= tol_h, ("entropy", r, g_en[r], o["entropy"][r])
        if vh and ns:
            g_v = val[sl].cpu().numpy().astype(np.float64)
            scale = np.max(np.abs(o["logits"]), axis=1)
            bad = np.abs(g_v - o["value"]) > rtol * (scale + np.abs(o["value"])) + 1e-5
            assert not bad.any(), ("value", np.argmax(bad), g_v[bad][:3], o["value"][bad][:3])
        self.rows_checked += ns
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
        if self.chains:
            gc = self.gpu.chain_state(self.e0, self.e1 - self.e0)
            oc = self.orc.chain_state()
            np.testing.assert_array_equal(gc["pending_count"], oc["pending_count"], err_msg=ctx)
            np.testing.assert_array_equal(gc["pending"], oc["pending"], err_msg=ctx)
            np.testing.assert_array_equal(gc["slot_chain"], oc["slot_chain"], err_msg=ctx)
            ql = np.asarray(g["qlen"])
            for e in range(ql.shape[0]):
                for m in range(ql.shape[1]):
                    n = int(ql[e, m])
                    np.testing.assert_array_equal(gc["queue_chain"][e, m, :n], oc["queue_chain"][e, m, :n],
                                                  err_msg=f"{ctx} queue chain ({e},{m})")
            np.testing.assert_array_equal(g["q_done"], oc["q_done"], err_msg=ctx)
            np.testing.assert_array_equal(g["q_met"], oc["q_met"], err_msg=ctx)
        if invariants:
            check_invariants(g, self.cfg, ctx=ctx)
        return g

    def close(self):
        self.gpu.close()
