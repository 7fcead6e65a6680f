"""GPU: im_tick_noalloc (actions staged in the library's static device array)
against im_tick (actions staged in the pool's own buffer), through the C ABI.

Two pools built from the same seeded inputs take the same ticks, one through
each entry point; the whole integer state (queues, slots, counters, chain
words and pending calls for chain pools) must agree bit for bit after every
call, including two calls in a row where the second has fewer rows than the
first, an empty tick, and pools of two shapes sharing the one static array.
A tick with more rows than the static array holds is refused with
IM_EINVAL before any work."""
import ctypes

import numpy as np
import pytest

import workload
from gpu_util import need_gpu, note
from helpers import assert_state_equal

pytestmark = pytest.mark.gpu


def _pool(cfg, seed, Q):
    torch = need_gpu()
    import paper_2606_11440_amd as P
    W, b = workload.gen.weights(cfg, seed, 0.1)
    table, _ = workload.gen.embedding(cfg, seed, rows=Q)
    cap = workload.gen.capacities(cfg, seed)
    emb = torch.from_numpy(table.view(np.int16) if cfg["dtype"] == "bf16" else table).cuda()
    return P.Pool(cfg, W, b, emb, cap, workload.gen.logit_bias(cfg)), emb


@pytest.mark.parametrize("name,over", [("c2", dict(E=300, lam=48.0)), ("c2c", dict(E=160, lam=8.0)),
                                       ("c1", dict(E=64))])
def test_tick_noalloc_equals_tick(name, over):
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get(name, T=8, **over)
    seed, Q = 70, 512
    note(f"[tick_noalloc] {name} E={cfg['E']}")
    a, ea = _pool(cfg, seed, Q)
    b, eb = _pool(cfg, seed, Q)
    counts = workload.gen.counts(cfg, seed)
    chains = cfg.get("max_steps", 1) > 1
    # the second call has fewer rows than the first; an empty tick later on
    for t, scale in enumerate((1.0, 0.3, 1.0, 0.0, 0.6, 1.0)):
        c = np.floor(counts[t] * scale).astype(np.int32)
        arr = workload.gen.tick(cfg, seed, t, c, Q)
        dev = P.device_arrivals(arr)
        a.tick(dev)
        b.tick_noalloc(dev)
        torch.cuda.synchronize()
        assert_state_equal(b.state(), a.state(), ctx=f"{name} t={t} rows={int(c.sum())}")
        if chains:
            ca, cb = a.chain_state(), b.chain_state()
            for k in ("queue_chain", "slot_chain", "pending", "pending_count"):
                np.testing.assert_array_equal(cb[k], ca[k], err_msg=f"{name} t={t} {k}")
    assert a.error() == 0 and b.error() == 0
    a.close()
    b.close()


def test_tick_noalloc_refuses_more_rows_than_its_array():
    torch = need_gpu()
    import paper_2606_11440_amd as P
    cfg = workload.configs.get("c2", E=2, T=2, max_arrivals=1 << 21)
    p, emb = _pool(cfg, 71, 64)
    n = (1 << 21) + 1
    off = torch.tensor([0, n, n], dtype=torch.int32, device="cuda")   # never read: refused first
    small32 = torch.zeros(1, dtype=torch.int32, device="cuda")
    small16 = torch.ones(1, dtype=torch.int16, device="cuda")
    arr = P._lib.ImArrivals()
    arr.offsets, arr.q_idx = off.data_ptr(), small32.data_ptr()
    arr.budget, arr.base_svc = small16.data_ptr(), small16.data_ptr()
    arr.n_total = n
    st = P._lib.load().im_tick_noalloc(p.h, ctypes.byref(arr), None)
    assert st == P._lib.IM_EINVAL
    assert "2^21" in P.im_last_error(p.h)
    torch.cuda.synchronize()
    assert p.state()["t"] == 0 and p.error() == 0
    p.close()
