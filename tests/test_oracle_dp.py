"""Pins for the oracle's exact schedule (Sec. 3.2, Eq. 10-11): brute-force
enumeration of every reuse placement on <= 12 steps, hand-worked cases and
monotonicity properties."""
import numpy as np
import pytest

from oracle import budget, dp, planner
from paper_2608_16354_amd import inputs as I

S = 2.0 ** -40


def small_problem(rng, K=None, tie_heavy=True):
    K = int(rng.integers(2, 13)) if K is None else K
    H = int(rng.integers(1, 4))
    if tie_heavy:
        q = rng.integers(0, 4, size=(K - 1, H)).astype(np.float64) * S
    else:
        q = rng.uniform(0.0, 1e-2, size=(K - 1, H))
    legal = (rng.random(K) < 0.85).astype(np.uint8)
    seg = None
    if rng.random() < 0.4:
        seg = np.cumsum(rng.random(K) < 0.2).astype(np.int32)
    n_cap = int(rng.integers(0, K))
    total = int(q.sum() / S) if tie_heavy else int(q.sum() * 2 ** 40)
    tau = int(rng.integers(0, max(1, total) + 1))
    xy = np.zeros((3, 2))
    yaw = np.zeros(3)
    p = I.SchedProblem(K, H, n_cap, legal, seg, xy, yaw, 0.0, 0.0, 10.0, 1.0, 1e-6,
                       q, q.copy(), np.zeros_like(q), np.zeros_like(q), tau_q=tau)
    if rng.random() < 0.5 and K > 2:
        s = int(rng.integers(2, K))
        p = p.replace(start_step=s, spent_q=int(rng.integers(0, tau + 1)),
                      spent_n=int(rng.integers(0, n_cap + 1)))
    return p


@pytest.mark.parametrize("seed", range(6))
def test_dp_equals_brute_force(seed):
    rng = np.random.default_rng(seed)
    for _ in range(250):
        p = small_problem(rng, tie_heavy=bool(rng.random() < 0.7))
        a = dp.schedule(p)
        b = dp.brute_force(p)
        assert a.reuse == b.reuse, (p, a, b)
        assert (a.n_reuse, a.cost_q) == (b.n_reuse, b.cost_q)
        # the returned cost is the cost of the returned mask, within budget
        n, c = dp.mask_cost(p, a.tables, a.reuse)
        assert (n, c) == (a.n_reuse, a.cost_q) and c <= p.tau_q - p.spent_q


def test_workload_schedules_equal_brute_force_small_K():
    w = I.WORKLOADS["dit-tiny-f32"]
    for tau in (0, 2 * 10 ** 9, 5 * 10 ** 9, I.TAU_INF):
        p = I.scene_problem(w, w.motions[0], tau_q=tau)
        assert dp.schedule(p).reuse == dp.brute_force(p).reuse


def test_hand_worked_three_steps():
    # K = 3, H_max = 2, every increment 1: reusing steps 2 and 3 costs 2
    q = np.array([[1.0, 2.0], [1.0, 2.0]]) * S      # envelope 1, 2 -> increments 1, 1
    p = I.SchedProblem(3, 2, 2, np.ones(3, np.uint8), None, np.zeros((2, 2)), np.zeros(2),
                       0.0, 0.0, 1.0, 1.0, 1e-6, q, q, q * 0, q * 0, tau_q=2)
    s = dp.schedule(p)
    assert s.reuse == [0, 1, 1] and s.n_reuse == 2 and s.cost_q == 2
    # budget 1 allows one reuse; both placements cost 1; the tie goes to the
    # mask with a full step last
    s = dp.schedule(p.replace(tau_q=1))
    assert s.reuse == [0, 1, 0] and s.cost_q == 1
    # max age 1 forbids the two-step run
    s = dp.schedule(p.replace(h_max=1, q0=q[:, :1], q1=q[:, :1], d0=q[:, :1] * 0, d1=q[:, :1] * 0))
    assert s.n_reuse == 1


def test_monotone_in_budget_and_cap():
    rng = np.random.default_rng(7)
    for _ in range(60):
        p = small_problem(rng, K=int(rng.integers(4, 11)), tie_heavy=False)
        p = p.replace(start_step=1, spent_q=0, spent_n=0, n_cap=p.K - 1)
        prev = -1
        for tau in sorted({0, 1, 10 ** 6, 10 ** 8, 10 ** 9, 10 ** 10, I.TAU_INF}):
            n = dp.schedule(p.replace(tau_q=tau)).n_reuse
            assert n >= prev
            prev = n
        prev = -1
        for cap in range(p.K):
            n = dp.schedule(p.replace(n_cap=cap, tau_q=I.TAU_INF)).n_reuse
            assert n >= prev and n <= cap
            prev = n


def test_degenerate_cases():
    w = I.WORKLOADS["dit-30x1920-bf16"]
    p = I.scene_problem(w, w.motions[0])
    assert dp.schedule(p.replace(tau_q=0)).n_reuse == 0          # positive costs, no budget
    assert dp.schedule(p.replace(n_cap=0)).n_reuse == 0
    s = dp.schedule(p)                                           # tau = infinity
    assert s.reuse[0] == 0                                       # first step always full
    # runs never exceed the maximum age
    run = 0
    for r in s.reuse:
        run = run + 1 if r else 0
        assert run <= w.h_max
    # unsupported scene -> full inference
    q = I.scene_problem(w, I.Motion(25.0, 0.0))
    assert dp.schedule(q).reuse == [0] * w.K
    # illegal steps are never reused
    legal = np.ones(w.K, np.uint8)
    legal[10:20] = 0
    s = dp.schedule(p.replace(legal=legal))
    assert sum(s.reuse[10:20]) == 0 and s.n_reuse > 0


def test_segments_block_cross_boundary_runs():
    K = 10
    q = np.full((K - 1, 3), 1.0) * S
    seg = np.array([0, 0, 0, 0, 0, 1, 1, 1, 1, 1], np.int32)
    p = I.SchedProblem(K, 3, K - 1, np.ones(K, np.uint8), seg, np.zeros((2, 2)), np.zeros(2),
                       0.0, 0.0, 1.0, 1.0, 1e-6, q, q, q * 0, q * 0)
    s = dp.schedule(p)
    # step 6 opens a new segment, so it cannot reuse a cache refreshed in segment 0
    assert s.reuse[5] == 0
    assert s.reuse == dp.brute_force(p).reuse


def test_budget_rule_targets_printed_counts():
    # Wan: 40 steps at 50 % -> 20 reuses (the A14B operating point reuses 0 + 20);
    # Epona: 100 steps at 60 % -> 60
    assert budget.target_reuses(0.5, 40) == 20
    assert budget.target_reuses(0.6, 100) == 60


def test_budget_rule_is_smallest_threshold_reaching_the_median():
    rng = np.random.default_rng(3)
    w = I.WORKLOADS["dit-tiny-f32"]
    motions = [I.Motion(float(rng.uniform(0, 20)), float(rng.uniform(-0.3, 0.3))) for _ in range(6)]
    probs = [I.scene_problem(w, m).replace(n_cap=w.K - 1) for m in motions]
    tau = budget.select_tau(probs, 0.5)
    target = budget.target_reuses(0.5, w.K)

    def median(t):
        b = sorted(dp.brute_force(p.replace(tau_q=t)).n_reuse for p in probs)
        return (b[2] + b[3]) / 2

    assert median(tau) >= target
    assert median(tau - 1) < target
