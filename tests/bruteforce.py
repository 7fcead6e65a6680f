"""A third, list-based model of the schedule step for tiny pools.

Written independently of the oracle: Python lists, `sorted` on (key, id)
tuples and a single pass per model. Used to cross-check the oracle (and the
GPU library) by exhaustive enumeration of forced actions on tiny pools.
Rules: action decode (Sec. 3), deadline-ordered service (Sec. 4.3), bounded
concurrency (Table 5), EMA latency (Sec. 5.4), with the documented readings."""
from __future__ import annotations

import copy


class TinyPool:
    def __init__(self, M, K, qcap, caps, key_mode="slack", max_slots=None):
        self.M, self.K, self.qcap, self.key_mode = M, K, qcap, key_mode
        self.S = max(caps) if max_slots is None else max_slots
        self.caps = list(caps)
        self.t = 0
        self.next_id = 0
        self.queues = [[] for _ in range(M)]          # lists of dicts, kept sorted
        self.slots = [[None] * self.S for _ in range(M)]
        self.ewma = [0] * M
        self.cnt = {k: [0] * M for k in ("rej_overflow", "enqueued", "started", "completed",
                                         "slo_met", "lat_sum", "wait_sum")}
        self.arrived = 0
        self.rej_nomodel = 0
        self.hist = [0] * (M * K)

    def clone(self):
        return copy.deepcopy(self)

    def _key(self, budget, svc):
        if self.key_mode == "deadline":
            return self.t + budget
        if self.key_mode == "fcfs":
            return self.t
        return self.t + budget - svc

    def step(self, reqs):
        """reqs: list of (budget, base_svc, action) in arrival order."""
        t = self.t
        self.arrived += len(reqs)
        per_model = {m: [] for m in range(self.M)}
        for i, (budget, base_svc, a) in enumerate(reqs):
            rid = self.next_id + i
            if a < 0:
                self.rej_nomodel += 1
                continue
            self.hist[a] += 1
            m, d = divmod(a, self.K)
            svc = base_svc * (d + 1)
            per_model[m].append(dict(key=self._key(budget, svc), id=rid, t_arr=t,
                                     svc=svc, budget=budget))
        for m in range(self.M):
            free = self.qcap - len(self.queues[m])
            take, drop = per_model[m][:max(free, 0)], per_model[m][max(free, 0):]
            self.cnt["rej_overflow"][m] += len(drop)
            self.cnt["enqueued"][m] += len(take)
            self.queues[m] = sorted(self.queues[m] + take, key=lambda r: (r["key"], r["id"]))
        for m in range(self.M):
            for s in range(self.caps[m]):
                if self.slots[m][s] is None and self.queues[m]:
                    r = self.queues[m].pop(0)
                    self.slots[m][s] = dict(r, rem=r["svc"])
                    self.cnt["started"][m] += 1
                    self.cnt["wait_sum"][m] += t - r["t_arr"]
            for s in range(self.S):
                r = self.slots[m][s]
                if r is None:
                    continue
                r["rem"] -= 1
                if r["rem"] == 0:
                    lat = t - r["t_arr"] + 1
                    self.ewma[m] += (lat * 256 - self.ewma[m]) // 8
                    self.cnt["completed"][m] += 1
                    self.cnt["lat_sum"][m] += lat
                    self.cnt["slo_met"][m] += int(lat <= r["budget"])
                    self.slots[m][s] = None
        self.next_id += len(reqs)
        self.t += 1

    def snapshot(self):
        """Same field names as the oracle's state() for env 0."""
        out = dict(t=self.t, next_id=self.next_id, arrived=self.arrived,
                   rej_nomodel=self.rej_nomodel, hist=list(self.hist),
                   ewma=list(self.ewma), qlen=[len(q) for q in self.queues],
                   backlog=[sum(r["svc"] for r in q) for q in self.queues],
                   busy=[sum(x is not None for x in sl) for sl in self.slots])
        out.update({k: list(v) for k, v in self.cnt.items()})
        out["queues"] = [[[r["key"], r["id"], r["t_arr"], r["svc"], r["budget"]] for r in q]
                         for q in self.queues]
        out["slots"] = [[[-1, 0, 0, 0] if r is None else [r["id"], r["t_arr"], r["rem"], r["budget"]]
                         for r in sl] for sl in self.slots]
        return out
