"""Oracle special cases that reduce to textbook routines.

* One model, c servers: the tick reduces to a discrete-time M/G/c station with
  a priority queue; checked against a heapq simulator written from scratch.
* FCFS key mode: every queue is FIFO by id (the Table 3 ablation baseline).
* Deadline key mode with equal budgets: FIFO as well (deadline = t + const).
* Deadline key mode: keys equal t_arrive + budget (Sec. 4.3)."""
import heapq

import numpy as np
import pytest

import oracle
from helpers import tiny_cfg


class HeapStation:
    """Discrete-time single-model station, c slots, priority by (key, id)."""

    def __init__(self, c, slots, mode):
        self.c, self.S, self.mode = c, slots, mode
        self.heap = []
        self.serving = [None] * slots
        self.t = 0
        self.nid = 0
        self.ewma = 0
        self.done = []          # (id, start, finish)
        self.start_of = {}
        self.arr_of = {}

    def step(self, reqs):
        t = self.t
        for budget, svc in reqs:
            key = {"slack": t + budget - svc, "deadline": t + budget, "fcfs": t}[self.mode]
            heapq.heappush(self.heap, (key, self.nid, t, svc, budget))
            self.arr_of[self.nid] = t
            self.nid += 1
        for s in range(self.c):
            if self.serving[s] is None and self.heap:
                key, rid, ta, svc, budget = heapq.heappop(self.heap)
                self.serving[s] = [rid, ta, svc, budget]
                self.start_of[rid] = t
        for s in range(self.S):
            job = self.serving[s]
            if job is None:
                continue
            job[2] -= 1
            if job[2] == 0:
                lat = t - job[1] + 1
                self.ewma += (256 * lat - self.ewma) // 8
                self.done.append((job[0], self.start_of[job[0]], t))
                self.serving[s] = None
        self.t += 1


@pytest.mark.parametrize("c,mode", [(1, "slack"), (2, "slack"), (3, "slack"), (1, "deadline"),
                                    (2, "fcfs")])
def test_single_model_matches_heap_station(c, mode):
    cfg = tiny_cfg(M=1, K=1, qcap=10_000, cap_hi=3, key_mode=mode, budget_hi=60)
    W = [np.zeros((8, cfg["feat_dim"]), np.float32), np.zeros((1, 8), np.float32)]
    b = [np.zeros(8, np.float32), np.zeros(1, np.float32)]
    o = oracle.Oracle(cfg, W, b, np.zeros((1, cfg["embed_dim"]), np.float32),
                      np.array([[c]], np.int32))
    hs = HeapStation(c, cfg["max_slots"], mode)
    rng = np.random.default_rng(c)
    for t in range(300):
        n = int(rng.poisson(0.9 * c / 3.0)) if t < 250 else 0
        reqs = [(int(rng.integers(1, 60)), int(rng.integers(1, 6))) for _ in range(n)]
        arr = dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32),
                   budget=np.array([r[0] for r in reqs], np.int16),
                   base_svc=np.array([r[1] for r in reqs], np.int16))
        o.schedule(arr, np.zeros(n, np.int32))
        hs.step(reqs)
        s = o.state()
        assert s["qlen"][0, 0] == len(hs.heap)
        assert s["ewma"][0, 0] == hs.ewma
        assert s["completed"][0, 0] == len(hs.done)
        q = s["queues"][0, 0, :len(hs.heap)]
        assert [tuple(r[:2]) for r in q] == [h[:2] for h in sorted(hs.heap)]
        busy_ids = sorted(j[0] for j in hs.serving if j is not None)
        assert sorted(x for x in s["slots"][0, 0, :, 0] if x >= 0) == busy_ids
    s = o.state()
    lat_sum = sum(f - hs.arr_of[rid] + 1 for rid, st, f in hs.done)
    wait_sum = sum(st - hs.arr_of[rid] for rid, st in hs.start_of.items())
    assert s["started"][0, 0] == len(hs.start_of)
    assert s["completed"][0, 0] == len(hs.done) and s["qlen"][0, 0] == 0
    assert s["lat_sum"][0, 0] == lat_sum and s["wait_sum"][0, 0] == wait_sum


@pytest.mark.parametrize("mode,equal_budget", [("fcfs", False), ("deadline", True)])
def test_fifo_modes(mode, equal_budget):
    cfg = tiny_cfg(M=2, K=2, qcap=500, cap_hi=1, key_mode=mode)
    W = [np.zeros((8, cfg["feat_dim"]), np.float32), np.zeros((4, 8), np.float32)]
    b = [np.zeros(8, np.float32), np.zeros(4, np.float32)]
    o = oracle.Oracle(cfg, W, b, np.zeros((1, cfg["embed_dim"]), np.float32),
                      np.array([[1, 1]], np.int32))
    rng = np.random.default_rng(3)
    for t in range(80):
        n = int(rng.integers(0, 5))
        bud = np.full(n, 9, np.int16) if equal_budget else rng.integers(1, 30, n).astype(np.int16)
        arr = dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32), budget=bud,
                   base_svc=rng.integers(1, 5, n).astype(np.int16))
        o.schedule(arr, rng.integers(0, 4, n).astype(np.int32))
        s = o.state()
        for m in range(2):
            q = s["queues"][0, m, :s["qlen"][0, m]]
            assert np.all(np.diff(q[:, 1]) > 0), "queue not FIFO by id"
            if mode == "deadline":
                assert np.all(q[:, 0] == q[:, 2] + q[:, 4])


def test_deadline_keys_are_arrival_plus_budget():
    cfg = tiny_cfg(M=1, K=3, qcap=500, cap_hi=1, key_mode="deadline")
    W = [np.zeros((8, cfg["feat_dim"]), np.float32), np.zeros((3, 8), np.float32)]
    b = [np.zeros(8, np.float32), np.zeros(3, np.float32)]
    o = oracle.Oracle(cfg, W, b, np.zeros((1, cfg["embed_dim"]), np.float32), np.array([[1]], np.int32))
    rng = np.random.default_rng(4)
    for t in range(40):
        n = 3
        arr = dict(offsets=np.array([0, n], np.int32), q_idx=np.zeros(n, np.int32),
                   budget=rng.integers(1, 30, n).astype(np.int16),
                   base_svc=rng.integers(1, 5, n).astype(np.int16))
        o.schedule(arr, rng.integers(0, 3, n).astype(np.int32))
    s = o.state()
    q = s["queues"][0, 0, :s["qlen"][0, 0]]
    assert np.all(q[:, 0] == q[:, 2] + q[:, 4])
    keys = [tuple(r[:2]) for r in q]
    assert keys == sorted(keys)
