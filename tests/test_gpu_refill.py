"""GPU parity where model queues keep running their sorted front dry over long
unsorted pools, so that the refill's top-64 selection runs many times per
queue, over pools from a few chunks of 64 entries to a few thousand entries.

Eight service slots per model with base service 1 tick start ~4 requests per
model and tick. With arrival-order keys (FCFS), a newcomer is never below the
front's largest key, so the front only shrinks by pops and every 64 pops are
followed by a refill from the whole pool (growing by ~9 entries per tick
until the queue fills); with slack keys the pool order is random, so the scan
keeps collecting candidates below its running threshold and merges them.
Lockstep with the oracle, integer state bit-exact (the queue contents in
order, the slots, the counters), single-step and chain pools."""
import pytest

import workload
from gpu_util import Pair, note

pytestmark = pytest.mark.gpu

FAST = dict(cap_lo=8, cap_hi=8, svc_mu=0.0, svc_sigma=0.0)
CASES = [
    ("fcfs_qcap1536", "c2", dict(FAST, key_mode="fcfs", qcap=1536, lam=64.0)),
    ("slack_qcap1536", "c2", dict(FAST, qcap=1536, lam=64.0)),
    ("deadline_qcap384", "c2", dict(FAST, key_mode="deadline", qcap=384, lam=64.0)),
    ("chain_fcfs_qcap1024", "c2c", dict(FAST, key_mode="fcfs", qcap=1024, lam=24.0)),
]


@pytest.mark.parametrize("sid,base,over", CASES, ids=[c[0] for c in CASES])
def test_refill_lockstep(sid, base, over):
    cfg = workload.configs.get(base, E=4, T=160, **over)
    note(f"[refill_lockstep] {sid}")
    p = Pair(cfg, seed=41, Q=512)
    longest = 0
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 10 == 9:
            g = p.compare_state(ctx=f"{sid} t={t}")
            longest = max(longest, int(g["qlen"].max()))
    started = int(g["started"].max())
    note(f"  rows={p.rows_checked} near-tie flips={p.flips} longest queue={longest} most started={started}")
    # a queue's front holds 64 entries: more than 3 x 64 dispatches from a
    # queue longer than two chunks took several refills from a non-empty pool
    assert longest > 2 * 64 and started > 3 * 64
    assert p.gpu.error() == 0
    p.close()
