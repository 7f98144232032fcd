"""Host logic of the benchmark's run record (CPU): which threshold each drift check was
compared with, and the algorithmic byte and FLOP counts the roofline figures use."""
import numpy as np

import bench
from oracle import dp
from paper_2608_16354_amd import inputs as I


class _Api:
    """The one library call run_record makes, answered by the oracle's planner."""

    class _S:
        def __init__(self, dbar):
            self.dbar = np.asarray(dbar, np.float64)

    def dc_schedule_dp(self, p):
        t = dp.schedule(p).tables
        return self._S(np.asarray(t.dbar, np.float64).reshape(p.K - 1, p.h_max))


def test_run_record_thresholds_follow_the_runs():
    w = I.WORKLOADS["dit-tiny-f32"]
    p = I.scene_problem(w, w.motions[0], thr=0.045)
    # a hand-made realized mask: refresh 1, reuse 2 (age 1), vetoed check at 3 (age 2;
    # refresh), reuse 4 (age 1 of the run refreshed at 3), reuse 5 (age 2)
    realized = np.array([[0], [1], [0], [1], [1], [0], [0], [0], [0], [0]], np.uint8)
    drift = np.full((w.K, 1), np.nan)
    drift[1, 0], drift[2, 0], drift[3, 0], drift[4, 0] = 0.01, 0.05, 0.02, 0.03
    rec = bench.run_record(_Api(), w, [p], realized, drift, [(np.zeros(w.K), 1, 7)])
    sc = rec["scenes"][0]
    assert sc["mask"] == "0101100000" and sc["n_veto"] == 1 and sc["charge_q"] == 7
    dbar = _Api().dc_schedule_dp(p).dbar
    assert [c["k"] for c in sc["checks"]] == [2, 3, 4, 5]
    want = [dbar[0, 0], dbar[0, 1], dbar[2, 0], dbar[2, 1]]     # (j, h) = (1,1), (1,2), (3,1), (3,2)
    assert [c["threshold"] for c in sc["checks"]] == want
    for c in sc["checks"]:
        assert c["margin"] == c["threshold"] - c["drift"]
    assert sc["min_abs_margin"] == min(abs(c["margin"]) for c in sc["checks"])


def test_algorithmic_counts_at_the_bench_shape():
    m = I.WORKLOADS["dit-30x1920-bf16"].model
    # 4 N^2 d for attention, 24 N d^2 for the four GEMMs at MLP 4d (the bench shape: 17,776 x 1920)
    assert bench.attention_flops(m) == 4.0 * 17776 ** 2 * 1920
    assert bench.gemm_flops(m) == 24.0 * 17776 * 1920 ** 2
    hb = bench.hbm_bytes(m)
    assert hb["cache_store"] == 17550 * 1920 * 10
    assert hb["head_reuse"] == 17550 * 1920 * 6 + 2 * 4 * 16 * 13 * 60 * 90
    assert hb["drift"] == 17550 * 1920 * 6
