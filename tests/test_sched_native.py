"""The library's host schedule (C++) against the oracle and brute force, bit-exact."""
import numpy as np
import pytest

from oracle import budget, dp, planner
from paper_2608_16354_amd import api
from paper_2608_16354_amd import inputs as I
from tests.test_oracle_dp import small_problem


def _same(p):
    a = api.dc_schedule_dp(p)
    o = dp.schedule(p)
    assert a.reuse == o.reuse, (p, a.reuse, o)
    assert (a.n_reuse, a.cost_q) == (o.n_reuse, o.cost_q)
    t = o.tables
    assert a.in_support == t.supported
    assert (a.L, a.Theta, a.zL, a.zTh, a.D) == (t.L, t.Th, t.zL, t.zTh, t.D)    # bit-exact f64
    if p.K > 1:
        assert a.chat_q.tolist() == t.chat_q
        assert a.dbar.tolist() == t.dbar
    return a


@pytest.mark.parametrize("seed", range(4))
def test_random_small_problems_match_oracle_and_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(300):
        p = small_problem(rng, tie_heavy=bool(rng.random() < 0.7))
        a = _same(p)
        assert a.reuse == dp.brute_force(p).reuse


@pytest.mark.parametrize("name", list(I.WORKLOADS))
def test_workload_schedules_match_oracle(name):
    w = I.WORKLOADS[name]
    tau = I.TAU_INF
    if w.tau == "rule":
        cal = [I.scene_problem(w, m) for m in I.calibration_motions(32)]
        tau = api.dc_select_tau(cal, w.rho)
        assert tau == budget.select_tau(cal, w.rho)
    for m in I.scene_motions(w):
        p = I.scene_problem(w, m, tau_q=tau)
        _same(p)
        # every suffix replan a veto could trigger, with the charge spent so far
        plan = dp.schedule(p)
        C, n = 0, 0
        j, age = 1, 0
        for k in range(2, w.K + 1):
            if plan.reuse[k - 1]:
                age += 1
                C += plan.tables.cost(j, age)
                n += 1
                _same(p.replace(start_step=k, spent_q=C, spent_n=n))
            else:
                j, age = k, 0


def test_random_motions_and_poses_bit_exact():
    rng = np.random.default_rng(9)
    w = I.WORKLOADS["dit-30x1920-bf16"]
    for _ in range(200):
        m = I.Motion(float(rng.uniform(-1, 26)), float(rng.uniform(-0.5, 0.5)), float(rng.uniform(0, 4)))
        _same(I.scene_problem(w, m, tau_q=int(rng.integers(0, 10 ** 11))))
    # headings that wrap across +-pi many times
    p = I.scene_problem(w, I.Motion(5.0, 0.3))
    yaw = np.cumsum(rng.uniform(-3.0, 3.0, size=p.pose_yaw.size))
    _same(p.replace(pose_yaw=yaw))


def test_select_tau_random_calibration_sets():
    rng = np.random.default_rng(5)
    w = I.WORKLOADS["dit-tiny-f32"]
    for n in (1, 2, 5, 6):
        probs = [I.scene_problem(w, I.Motion(float(rng.uniform(0, 22)), float(rng.uniform(-0.35, 0.35))))
                 .replace(n_cap=w.K - 1) for _ in range(n)]
        for rho in (0.1, 0.5, 0.6, 0.9):
            assert api.dc_select_tau(probs, rho) == budget.select_tau(probs, rho)


def test_invalid_problems_are_rejected():
    w = I.WORKLOADS["dit-tiny-f32"]
    p = I.scene_problem(w, w.motions[0])
    for bad in (dict(h_max=0), dict(n_cap=w.K), dict(n_cap=-1), dict(tau_q=-1), dict(start_step=0),
                dict(start_step=w.K + 1), dict(spent_n=4)):
        with pytest.raises(api.L.DriveCacheError) as e:
            api.dc_schedule_dp(p.replace(**bad))
        assert e.value.code == api.L.DC_ERR_ARG
