"""The controller side of the Top-5 mixture (100 steps) and Top-3 drifting (200 steps) closed loops, pinned to the
oracle (Alg. 1; Eq. rapid-integral, rapid-delta, rapid-gate, rapid-update; Eq. vio).

Counts come from the oracle's own closed loop on each workload's synthetic
hidden states (the first 512 tokens of every step's batch, the workload's K
and E, ID Balancing with K_i = K_d = 6e-3 and centring): the oracle routes
each batch with its current bias, updates, and the counts it produced are
fed to the GPU's two stand-alone controller kernels -- the single-layer
update with MaxVio/MinVio (idb_controller_step) and the batched layers
kernel with its diagnostics (idb_controller_update_layers).  Every step's
bias, e_prev, step, status, MaxVio/MinVio and diagnostics must be the
oracle's bit for bit.  The drifting mixture moves the load from step to
step, so the derivative gate opens (Eq. rapid-gate), which is asserted.

The update run inside idb_router_step's slice merge is pinned over whole
trajectories in test_gpu_router_step_oracle.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39137_amd import binding as B
from paper_2609_39137_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
ROWS = 512


@pytest.mark.parametrize("name", ["top5-of-768-mixture", "top3-of-768-drift"])
def test_workload_loop_controller_matches_oracle(name):
    wl = synth.WORKLOADS[name]
    W = synth.router_weight(wl)
    Ki = Kd = 6e-3
    cfg = B.ControllerCfg(wl.E, Ki, Kd)
    ref = oracle.ControllerState(wl.E)
    one = B.ControllerState(wl.E, DEV)
    lay = B.ControllerState(wl.E, DEV, layers=1)
    stats1 = torch.empty(2, dtype=torch.float64, device=DEV)
    statsL = torch.empty((1, 2), dtype=torch.float64, device=DEV)
    diagL = torch.empty((1, 4), dtype=torch.float64, device=DEV)
    gates = []
    for t in range(wl.steps):
        x = synth.hidden_states(wl, step=t, rows=np.arange(ROWS))
        _, _, c = oracle.router(x, W, ref.bias, wl.K)
        want_stats = oracle.load_stats(c)
        status, want_diag = oracle.controller_diag(c, ref, Ki, Kd)
        assert status == oracle.STATUS_OK
        gates.append(want_diag[0])
        counts = torch.from_numpy(c).to(DEV)
        if t % 25 == 0:
            print(f"[loop] {name} step {t}", flush=True)
        B.idb_controller_step(counts, cfg, one, stats1)
        B.idb_controller_update_layers(counts.view(1, -1), cfg, lay, statsL, diagL)
        msg = f"{name} step {t}"
        for st, bias, e_prev in ((one, one.bias, one.e_prev), (lay, lay.bias[0], lay.e_prev[0])):
            np.testing.assert_array_equal(bias.cpu().numpy().view(np.uint32), ref.bias.view(np.uint32), err_msg=msg)
            np.testing.assert_array_equal(e_prev.cpu().numpy().view(np.uint32), ref.e_prev.view(np.uint32),
                                          err_msg=msg)
            assert int(st.step[0].item()) == t + 1 and int(st.status[0].item()) == 0, msg
        np.testing.assert_array_equal(stats1.cpu().numpy(), want_stats, err_msg=msg)
        np.testing.assert_array_equal(statsL.cpu().numpy()[0], want_stats, err_msg=msg)
        np.testing.assert_array_equal(diagL.cpu().numpy()[0], want_diag, err_msg=msg)
    assert gates[0] == 0.0 and max(gates[1:]) > 0.1, gates
