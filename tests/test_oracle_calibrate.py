"""Pins for the oracle's anchor calibration (Eq. 5-7): every tangent against central
finite differences of the float64 forward pass, the tail Jacobian-vector product
against re-running the perturbed sampler tail, and exact cases (a zero residual
gives zero responses; the tangent is linear)."""
import numpy as np
import pytest

from oracle import calibrate as cal
from oracle import dit, dp
from paper_2608_16354_amd import inputs as I

W_TINY = I.WORKLOADS["dit-tiny-f32"]


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.fixture(scope="module")
def tiny():
    w = W_TINY
    P = dit.Params(I.Weights(w.model, w.cfg_id))
    x1 = I.latent(w.model, 1).astype(np.float64)
    txt = I.text(w.model, 1).astype(np.float64)
    return w, P, x1, txt, I.sigmas(w.K)


@pytest.fixture(scope="module")
def trace(tiny):
    w, P, x1, txt, sig = tiny
    return cal.Trace(P, x1, txt, sig)


def test_layer_norm_and_modulate_tangents():
    rng = np.random.default_rng(1)
    x, dx = rng.standard_normal((6, 96)) * 3 + 1.5, rng.standard_normal((6, 96))
    sh, sc = rng.standard_normal(96), rng.standard_normal(96)
    h = 1e-6
    y, dy = cal.jvp_modulate(x, dx, sh, sc, 1e-6)
    fd = (dit.modulate(x + h * dx, sh, sc, 1e-6) - dit.modulate(x - h * dx, sh, sc, 1e-6)) / (2 * h)
    assert np.allclose(y, dit.modulate(x, sh, sc, 1e-6), rtol=0, atol=1e-13)
    assert _rel(dy, fd) < 1e-8


def test_gelu_tangent():
    z = np.linspace(-6, 6, 1001)
    dz = np.cos(z)
    g, dg = cal.jvp_gelu_tanh(z, dz)
    h = 1e-6
    fd = (dit.gelu_tanh(z + h * dz) - dit.gelu_tanh(z - h * dz)) / (2 * h)
    assert np.array_equal(g, dit.gelu_tanh(z))
    assert _rel(dg, fd) < 1e-8


def test_attention_tangent():
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((40, 32)) for _ in range(3))
    dq, dk, dv = (rng.standard_normal((40, 32)) for _ in range(3))
    o, do = cal.jvp_attention(q, k, v, dq, dk, dv, heads=4)
    h = 1e-6
    fd = (dit.attention(q + h * dq, k + h * dk, v + h * dv, 4)
          - dit.attention(q - h * dq, k - h * dk, v - h * dv, 4)) / (2 * h)
    assert np.allclose(o, dit.attention(q, k, v, 4), rtol=1e-12, atol=1e-12)
    assert _rel(do, fd) < 1e-8


def test_network_tangent(tiny):
    w, P, x1, txt, sig = tiny
    d = np.random.default_rng(3).standard_normal(x1.shape)
    mods, hm = dit.step_modulation(P, sig[3])

    def net(x):
        h_out = dit.backbone(P, mods, dit.embed(P, x, txt))
        return dit.head(P, hm, h_out[: w.model.n_v])

    v, dv = cal.jvp_network(P, sig[3], x1, d, txt)
    h = 1e-4
    fd = (net(x1 + h * d) - net(x1 - h * d)) / (2 * h)
    assert np.allclose(v, net(x1), rtol=0, atol=1e-12)
    assert _rel(dv, fd) < 1e-6


@pytest.mark.parametrize("t", [2, 6, 9])
def test_tail_jvp_against_rerunning_the_tail(trace, t):
    e = np.random.default_rng(t).standard_normal(trace.x_out.shape)
    e *= 1e-2 * np.linalg.norm(trace.v[t - 1]) / np.linalg.norm(e)
    g = cal.tail_jvp(trace, t, e)
    h = 1e-3
    fd = (cal.tail_rerun(trace, t, h * e) - cal.tail_rerun(trace, t, -h * e)) / (2 * h)
    assert _rel(g, fd) < 1e-6
    # the unperturbed rerun is the trace's own terminal latent
    assert np.allclose(cal.tail_rerun(trace, t, 0 * e), trace.x_out, rtol=0, atol=1e-12)


def test_tail_jvp_is_linear_exactly(trace):
    e = np.random.default_rng(5).standard_normal(trace.x_out.shape)
    assert np.array_equal(cal.tail_jvp(trace, 4, 2.0 * e), 2.0 * cal.tail_jvp(trace, 4, e))


def test_last_step_perturbation_moves_the_output_by_its_euler_step(trace):
    e = np.random.default_rng(6).standard_normal(trace.x_out.shape)
    K, s = trace.K, trace.sigmas
    assert np.array_equal(cal.tail_jvp(trace, K, e), (s[K] - s[K - 1]) * e)


def test_zero_residual_gives_zero_responses(tiny):
    w, _, x1, txt, sig = tiny
    Pz = dit.Params(I.Weights(w.model, w.cfg_id, zero_out=("w_o", "b_o", "w_2", "b_2")))
    tr = cal.Trace(Pz, x1, txt, sig)
    q, d = cal.run_tables(tr, 2, 1e-6)
    assert np.all(q == 0.0)
    assert np.all(d[:-1] > 0.0)           # the inputs still drift


def test_tables_shape_and_the_planner_on_calibrated_tables(tiny, trace):
    w, P, x1, txt, sig = tiny
    q0, d0 = cal.run_tables(trace, w.h_max, w.eps)
    tr1 = cal.Trace(P, I.latent(w.model, 1, 1).astype(np.float64), I.text(w.model, 1, 1).astype(np.float64), sig)
    q1, d1 = cal.run_tables(tr1, w.h_max, w.eps)
    K = w.K
    for q, d in ((q0, d0), (q1, d1)):
        assert q.shape == (K - 1, w.h_max) and np.all(q >= 0) and np.all(d >= 0)
        assert q[K - 2, 1] == 0.0 and d[K - 2, 1] == 0.0        # run past the last step
        assert np.all(q[: K - 2] > 0)
    # the planner on the calibrated tables: the library's schedule equals the oracle's bit for bit
    from paper_2608_16354_amd import api
    for m in (w.motions[0], I.Motion(2.0, 0.0), I.Motion(9.0, 0.2)):
        p = I.scene_problem(w, m).replace(q0=q0, q1=q1, d0=d0, d1=d1)
        plan = dp.schedule(p)
        a = api.dc_schedule_dp(p)
        assert a.reuse == plan.reuse and (a.n_reuse, a.cost_q) == (plan.n_reuse, plan.cost_q)
        assert a.chat_q.tolist() == plan.tables.chat_q and a.dbar.tolist() == plan.tables.dbar
