"""Pins for the oracle's causal controller and samplers (Sec. 3.2, Eq. 1, Eq. 12):
exact equalities the method guarantees, checked on the small fp32 workload."""
import numpy as np
import pytest

from oracle import dp, dit, runtime
from paper_2608_16354_amd import inputs as I

W_TINY = I.WORKLOADS["dit-tiny-f32"]


@pytest.fixture(scope="module")
def tiny():
    w = W_TINY
    W = I.Weights(w.model, w.cfg_id)
    return w, W, I.latent(w.model, 1), I.text(w.model, 1), I.sigmas(w.K)


@pytest.fixture(scope="module")
def uncached(tiny):
    w, W, x1, txt, sig = tiny
    return runtime.sample(W, x1, txt, sig, I.scene_problem(w, w.motions[0]), uncached=True)


def test_all_refresh_equals_uncached_exactly(tiny, uncached):
    w, W, x1, txt, sig = tiny
    # a zero threshold vetoes every planned reuse: every step refreshes
    res = runtime.sample(W, x1, txt, sig, I.scene_problem(w, w.motions[0], thr=0.0))
    assert sum(res.realized) == 0 and any(r.vetoed for r in res.records)
    assert np.array_equal(res.x, uncached.x)


def test_no_veto_executes_the_plan(tiny, uncached):
    w, W, x1, txt, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    res = runtime.sample(W, x1, txt, sig, p)
    assert res.realized == dp.schedule(p).reuse
    assert sum(res.realized) == 3            # the reuse cap of the tiny workload
    assert not np.array_equal(res.x, uncached.x)
    assert res.charge == dp.schedule(p).cost_q


def test_zero_residual_makes_every_schedule_exact(tiny):
    w, _, x1, txt, sig = tiny
    Wz = I.Weights(w.model, w.cfg_id, zero_out=("w_o", "b_o", "w_2", "b_2"))
    p = I.scene_problem(w, w.motions[0])
    a = runtime.sample(Wz, x1, txt, sig, p)
    b = runtime.sample(Wz, x1, txt, sig, p, uncached=True)
    assert sum(a.realized) == 3
    assert np.array_equal(a.x, b.x)


def test_reuse_step_is_input_plus_stored_residual(tiny):
    w, W, x1, txt, sig = tiny
    P = dit.Params(W)
    mods, _ = dit.step_modulation(P, sig[0])
    h_in = dit.embed(P, x1, txt)
    h_out = dit.backbone(P, mods, h_in)
    r = h_out[: w.model.n_v] - h_in[: w.model.n_v]
    # at the refresh step itself, h_in + r reproduces h_out to rounding
    assert np.allclose(h_in[: w.model.n_v] + r, h_out[: w.model.n_v], rtol=0, atol=1e-14)


def test_forced_veto_keeps_prefix_and_replans_suffix(tiny):
    w, W, x1, txt, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    plan = dp.schedule(p)
    first = plan.reuse.index(1) + 1                    # 1-based step of the first planned reuse
    res = runtime.sample(W, x1, txt, sig, p, force_veto=(first,))
    assert res.realized[: first - 1] == plan.reuse[: first - 1]
    assert res.realized[first - 1] == 0 and res.records[first - 1].vetoed
    # the suffix is the exact optimum of the replan problem (brute force), from age zero
    rp = p.replace(start_step=first, spent_q=0, spent_n=0)
    assert res.realized[first:] == dp.brute_force(rp).reuse[first:]


def test_mid_threshold_veto_replans_with_remaining_budget(tiny):
    w, W, x1, txt, sig = tiny
    p = I.scene_problem(w, w.motions[0], thr=0.045)
    res = runtime.sample(W, x1, txt, sig, p)
    vet = [r.k for r in res.records if r.vetoed]
    assert len(vet) >= 1 and len(res.plans) == 1 + len(vet)
    # every accepted reuse respected the threshold and every veto exceeded it
    for r in res.records:
        if r.drift is not None:
            assert (r.drift <= r.threshold + p.eps) == (not r.vetoed)
    # the charge never exceeds the budget, and equals the sum of accepted costs
    t = res.plans[0].tables
    C = sum(t.cost(r.j, r.age) for r in res.records if r.realized)
    assert C == res.charge


def test_drift_definitions():
    u = np.random.default_rng(1).normal(size=(10, 6))
    assert runtime.drift_value(runtime.drift_sums(u, u), 1e-6) == 0.0
    # zero reference: the relative L1 drift is S2 / (S2 + eps)
    s = runtime.drift_sums(u, np.zeros_like(u))
    assert runtime.drift_value(s, 1e-6) == pytest.approx(s[1] / (s[1] + 1e-6))
    # scale invariance up to eps
    a, b = runtime.drift_sums(u, 0.9 * u), runtime.drift_sums(7 * u, 6.3 * u)
    assert runtime.drift_value(a, 0.0) == pytest.approx(runtime.drift_value(b, 0.0), rel=1e-12)
    assert runtime.drift_value(a, 0.0, "l2") == pytest.approx(0.1, rel=1e-12)


def test_unsupported_scene_runs_uncached(tiny, uncached):
    w, W, x1, txt, sig = tiny
    res = runtime.sample(W, x1, txt, sig, I.scene_problem(w, I.Motion(30.0, 0.0)))
    assert sum(res.realized) == 0 and all(r.drift is None for r in res.records)
    assert np.array_equal(res.x, uncached.x)
