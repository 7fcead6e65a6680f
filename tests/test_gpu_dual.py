"""GPU parity of the dual update (im_dual_update, Eq. 7) and of the Q16 cost
counter it reads: lambda bit-exact with the oracle (both take the same
correctly rounded fp64 steps over exact integer sums), the cost counters
bit-exact in every state comparison; the closed-form ramp of a single-slot
FCFS model, a c2 workload with updates every few ticks (two sampled envs
followed by the oracle, all envs reduced on the GPU: so the oracle runs the
whole small pool here) and no-completion calls."""
import numpy as np
import pytest

import workload
from gpu_util import Pair, need_gpu, note

pytestmark = pytest.mark.gpu


def _lam(torch, v):
    return torch.tensor([v], dtype=torch.float64, device="cuda")


def test_dual_closed_form_ramp():
    torch = need_gpu()
    from helpers import tiny_cfg
    cfg = tiny_cfg(M=1, K=1, widths=[32, 1], key_mode="fcfs", qcap=16, cap_hi=1, T=200)
    note("[dual_ramp]")
    p = Pair(cfg, seed=1, Q=4)
    lam_g, lam_o = _lam(torch, 0.2), 0.2
    for t in range(cfg["T"]):
        if t % 5 == 0:
            arr = dict(offsets=np.array([0, 1], np.int32), q_idx=np.array([0], np.int32),
                       budget=np.array([8], np.int16), base_svc=np.array([4], np.int16))
        else:
            z = np.zeros(0, np.int32)
            arr = dict(offsets=np.array([0, 0], np.int32), q_idx=z, budget=z.astype(np.int16),
                       base_svc=z.astype(np.int16))
        p.step(arr)
        if t % 10 == 9:
            p.gpu.dual_update(0.001, 1.0, lam_g)
            lam_o = p.orc.dual_update(lam_o, 0.001, 1.0)
            torch.cuda.synchronize()
            assert lam_g.item() == lam_o, (t, lam_g.item(), lam_o)
    assert lam_o == pytest.approx(0.2 - 20 * 0.0005, abs=1e-12)
    p.compare_state(ctx="ramp end")
    p.close()


@pytest.mark.parametrize("name,E", [("c2", 6), ("c4", 8)])
def test_dual_matches_oracle(name, E):
    torch = need_gpu()
    cfg = workload.configs.get(name, E=E, T=50)
    note(f"[dual_matches_oracle] {name} E={E}")
    p = Pair(cfg, seed=31, Q=256)
    lam_g, lam_o = _lam(torch, 0.3), 0.3
    for t in range(cfg["T"]):
        p.step(p.arrivals(t))
        if t % 7 == 6:
            for _ in range(2):                 # the second call has no new completions
                p.gpu.dual_update(0.05, 0.9, lam_g)
                lam_o = p.orc.dual_update(lam_o, 0.05, 0.9)
            torch.cuda.synchronize()
            assert lam_g.item() == lam_o, (t, lam_g.item(), lam_o)
            p.compare_state(ctx=f"{name} t={t}")
    p.close()
