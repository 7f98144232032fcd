"""Pins for the oracle's model-specific legality variants (Sec. 3.2, last paragraph;
Table 4): two experts split at a step with no cache crossing the switch, and
guidance branches with separate caches.  Each is tied to the single-branch,
single-expert sampler by an equality the combination rule or the weights make
exact, on the small fp32 workload."""
import numpy as np
import pytest

from oracle import dp, runtime
from paper_2608_16354_amd import inputs as I

W_TINY = I.WORKLOADS["dit-tiny-f32"]
K_SWITCH = 6


@pytest.fixture(scope="module")
def tiny():
    w = W_TINY
    W = I.Weights(w.model, w.cfg_id)
    txt_null = I.text(w.model, 1, scene=7)
    return w, W, I.latent(w.model, 1), I.text(w.model, 1), txt_null, I.sigmas(w.K)


def _segmented(w, k_switch=K_SWITCH, **kw):
    p = I.scene_problem(w, w.motions[0], **kw)
    seg = np.array([0] * (k_switch - 1) + [1] * (w.K - k_switch + 1), np.int32)
    return p.replace(segment=seg)


def test_guidance_one_is_the_conditional_sample(tiny):
    w, W, x1, txt, txt_null, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    plain = runtime.sample(W, x1, txt, sig, p)
    g1 = runtime.sample(W, x1, txt, sig, p, guidance=1.0, txt_null=txt_null)
    assert g1.realized == plain.realized and sum(plain.realized) > 0
    # v_u + 1 (v_c - v_u) differs from v_c by rounding only
    assert np.max(np.abs(g1.x - plain.x)) <= 1e-12 * np.max(np.abs(plain.x))


def test_guidance_zero_is_the_unconditional_sample(tiny):
    w, W, x1, txt, txt_null, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    g0 = runtime.sample(W, x1, txt, sig, p, guidance=0.0, txt_null=txt_null)
    un = runtime.sample(W, x1, txt_null, sig, p)
    # v = v_u + 0 (v_c - v_u) = v_u exactly; the decisions depend on the video rows only
    assert g0.realized == un.realized
    assert np.array_equal(g0.x, un.x)


@pytest.mark.parametrize("wg", [0.5, 3.0])
def test_identical_branches_make_guidance_exact(tiny, wg):
    w, W, x1, txt, _, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    plain = runtime.sample(W, x1, txt, sig, p)
    same = runtime.sample(W, x1, txt, sig, p, guidance=wg, txt_null=txt)
    assert np.array_equal(same.x, plain.x)


def test_guidance_branches_keep_separate_caches(tiny):
    """With both branches cached the plan's reuses execute, and the guided result stays
    near full-evaluation guidance (caching approximates; it does not fall apart)."""
    w, W, x1, txt, txt_null, sig = tiny
    p = I.scene_problem(w, w.motions[0])
    wg = 3.0
    cached = runtime.sample(W, x1, txt, sig, p, guidance=wg, txt_null=txt_null)
    full = runtime.sample(W, x1, txt, sig, p, guidance=wg, txt_null=txt_null, uncached=True)
    assert sum(cached.realized) == 3
    # caching changes the result (it is an approximation) but stays close to full guidance
    err = np.linalg.norm(cached.x - full.x) / np.linalg.norm(full.x)
    assert 0.0 < err < 0.5


def test_same_weights_as_both_experts_is_the_segmented_sample(tiny):
    w, W, x1, txt, _, sig = tiny
    p = _segmented(w)
    plain = runtime.sample(W, x1, txt, sig, p)
    two = runtime.sample(W, x1, txt, sig, p, W_low=I.Weights(w.model, w.cfg_id), k_switch=K_SWITCH)
    assert two.realized == plain.realized
    assert np.array_equal(two.x, plain.x)


def test_no_reuse_run_crosses_the_expert_switch(tiny):
    w, W, x1, txt, _, sig = tiny
    W_low = I.Weights(w.model, w.cfg_id + 50)
    p = _segmented(w)
    res = runtime.sample(W, x1, txt, sig, p, W_low=W_low, k_switch=K_SWITCH)
    assert res.records[K_SWITCH - 1].realized == 0          # the switch step evaluates
    for r in res.records:
        if r.realized:
            assert (r.j >= K_SWITCH) == (r.k >= K_SWITCH)     # the run's refresh step is on its side
    # the low-noise expert really runs: with its weights swapped for the high one's the result moves
    assert not np.array_equal(res.x, runtime.sample(W, x1, txt, sig, p).x)
    # and a plan that would cross is rejected up front
    with pytest.raises(ValueError):
        runtime.sample(W, x1, txt, sig, I.scene_problem(w, w.motions[0]), W_low=W_low, k_switch=K_SWITCH)


def test_segment_change_removes_reuse_at_the_switch():
    w = W_TINY
    p = _segmented(w, thr=I.NO_VETO)
    plan = dp.schedule(p).reuse
    assert plan[K_SWITCH - 1] == 0
