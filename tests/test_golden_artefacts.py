"""The stored oracle samples (tests/golden/oracle_*.npz) against the controller of
Sec. 3.2 and the planner, on the CPU.  Whatever wrote a file, its decisions must follow
from its own drifts, thresholds and budget: a drift check runs exactly on the planned
reuses (Eq. 12), a planned reuse is executed iff its drift is within the threshold and
vetoed otherwise, and without a veto the realized mask is the exact DP plan (Eq. 10-11)
of the workload's problem.  A file written from other inputs is refused by its
fingerprint."""
import glob
import os

import numpy as np
import pytest

from oracle import budget, dp
from paper_2608_16354_amd import inputs as I

HERE = os.path.dirname(os.path.abspath(__file__))
FILES = sorted(glob.glob(os.path.join(HERE, "golden", "oracle_*.npz")))


@pytest.mark.parametrize("path", FILES, ids=[os.path.basename(f) for f in FILES])
def test_stored_sample_follows_the_controller(path):
    z = np.load(path, allow_pickle=False)
    w = I.WORKLOADS[str(z["workload"])]
    assert str(z["fingerprint"]) == I.input_fingerprint(w)
    S = int(z["steps"])
    assert 1 <= S <= w.K
    for key in ("realized", "planned", "vetoed", "drift", "drift_l2", "threshold"):
        assert len(z[key]) == S, key
    assert len(z["plan"]) == w.K
    cal = [I.scene_problem(w, m) for m in I.calibration_motions(32)]
    tau = budget.select_tau(cal, w.rho)
    assert int(z["tau_q"]) == tau
    thr = float(z["thr"])
    p = I.scene_problem(w, w.motions[0], tau_q=tau, thr=thr)

    realized, planned, vetoed = (z[k].astype(bool) for k in ("realized", "planned", "vetoed"))
    drift, drift_l2, threshold = z["drift"], z["drift_l2"], z["threshold"]
    assert not planned[0]                                   # the first step evaluates the backbone
    checked = ~np.isnan(drift)
    assert np.array_equal(checked, planned)                 # a check on exactly the planned reuses
    assert np.array_equal(checked, ~np.isnan(drift_l2))
    assert np.all(threshold[checked] == thr)                # constant anchor drift tables
    within = drift[checked] <= threshold[checked] + p.eps
    assert np.array_equal(realized[checked], within)        # executed iff within the threshold
    assert np.array_equal(vetoed[checked], ~within)         # vetoed otherwise
    assert not np.any(realized[~checked] | vetoed[~checked])
    assert int(z["n_veto"]) == int(vetoed.sum())
    assert np.all((drift[checked] >= 0) & (drift_l2[checked] >= 0))
    # the final plan keeps every executed step's planned flag (a replan rewrites only the
    # steps after the vetoed one)
    assert np.array_equal(z["plan"][:S].astype(bool), planned)
    if int(z["n_veto"]) == 0:
        plan = dp.schedule(p)
        assert realized.astype(int).tolist() == plan.reuse[:S]
        assert z["plan"].astype(int).tolist() == plan.reuse
    x = z["x"]
    assert x.shape == (w.model.lat_c, w.model.lat_t, w.model.lat_h, w.model.lat_w)
    assert np.all(np.isfinite(x))
