"""Oracle pinned by closed-form invariants on every tick of seeded runs of
each workload (reduced env counts): request conservation, sorted queues,
capacity bounds, backlog accounting, key formulas, work conservation."""
import numpy as np
import pytest

import workload
from helpers import check_invariants, make_oracle


@pytest.mark.parametrize("name,E,T,mode", [("c0", 1, 100, "slack"), ("c1", 4, 60, "slack"),
                                           ("c2", 4, 40, "deadline"), ("c3", 2, 30, "slack"),
                                           ("c4", 6, 40, "fcfs")])
def test_invariants_every_tick(name, E, T, mode):
    cfg = workload.configs.get(name, E=E, T=T, key_mode=mode)
    Q = 256
    o, _ = make_oracle(cfg, seed=5, Q=Q)
    cnt = workload.gen.counts(cfg, 5)
    prev = o.state()
    for t in range(T):
        arr = workload.gen.tick(cfg, 5, t, cnt[t], Q)
        o.tick(arr)
        s = o.state()
        check_invariants(s, cfg, prev, ctx=f"{name} t={t}")
        prev = s
    assert o.error == 0
    if name == "c4":
        assert s["rej_overflow"].sum() > 0      # the overload case overflows


def test_invariants_with_outage_and_scale_down():
    """Host knobs mid-run: a disabled model receives nothing new; a model
    scaled to c=0 drains its slots and is never routed to."""
    cfg = workload.configs.get("c0", T=80)
    o, _ = make_oracle(cfg, seed=6, Q=64)
    cnt = workload.gen.counts(cfg, 6)
    prev = o.state()
    for t in range(80):
        if t == 20:
            o.set_enabled(0, 1, 0)
            o.set_capacity(0, 2, 0)
        arr = workload.gen.tick(cfg, 6, t, cnt[t], 64)
        act = o.tick(arr)
        if t >= 20:
            assert not np.any((act // cfg["K"] == 1) | (act // cfg["K"] == 2))
        s = o.state()
        check_invariants(s, cfg, prev, ctx=f"t={t}")
        prev = s
    assert s["busy"][0, 2] == 0
