"""Pins for the oracle's generator pieces: closed forms, special cases that
reduce to library routines, and invariants."""
import math

import numpy as np
import pytest
import scipy.special

from oracle import dit
from paper_2608_16354_amd import inputs as I

rng = np.random.default_rng(11)


def test_layer_norm_moments_and_constant_rows():
    x = rng.normal(3.0, 2.0, size=(7, 64))
    y = dit.layer_norm(x, 1e-6)
    assert np.allclose(y.mean(axis=1), 0.0, atol=1e-13)
    var = x.var(axis=1)
    assert np.allclose(y.var(axis=1), var / (var + 1e-6), rtol=1e-12)
    assert np.array_equal(dit.layer_norm(np.full((2, 8), 5.0), 1e-6), np.zeros((2, 8)))
    # zero shift and scale give the plain normalisation
    assert np.array_equal(dit.modulate(x, np.zeros(64), np.zeros(64), 1e-6), y)


def test_activations():
    z = np.linspace(-8, 8, 101)
    assert dit.gelu_tanh(np.array([0.0]))[0] == 0.0
    # tanh-GELU: g(z) - g(-z) = z exactly in real arithmetic
    assert np.allclose(dit.gelu_tanh(z) - dit.gelu_tanh(-z), z, atol=1e-14)
    # tends to the identity / zero in the tails; stays within 0.02 of erf-GELU
    assert abs(dit.gelu_tanh(np.array([20.0]))[0] - 20.0) < 1e-12
    erf_gelu = 0.5 * z * (1 + scipy.special.erf(z / math.sqrt(2)))
    assert np.max(np.abs(dit.gelu_tanh(z) - erf_gelu)) < 2e-3
    assert np.allclose(dit.silu(z), z * scipy.special.expit(z), rtol=1e-14, atol=1e-300)


def test_timestep_features_at_zero_and_period():
    e = dit.timestep_features(0.0)
    assert np.array_equal(e, np.concatenate([np.ones(128), np.zeros(128)]))
    e = dit.timestep_features(2 * math.pi)
    # the slowest... and the fastest frequency (w_0 = 1) completes a full period
    assert e[0] == pytest.approx(1.0) and e[128] == pytest.approx(0.0, abs=1e-12)
    assert np.allclose(e[:128] ** 2 + e[128:] ** 2, 1.0)


def test_attention_special_cases():
    N, dh = 9, 8
    k = rng.normal(size=(N, dh))
    v = rng.normal(size=(N, dh))
    # zero queries attend uniformly: every output row is the mean of the values
    o = dit.attention_rows(np.zeros((3, dh)), k, v)
    assert np.allclose(o, v.mean(axis=0)[None, :], atol=1e-14)
    # a single key returns its value
    assert np.allclose(dit.attention_rows(rng.normal(size=(2, dh)), k[:1], v[:1]), v[:1], atol=1e-14)
    # a dominant logit selects its value
    q = np.zeros((1, dh))
    q[0, 0] = 1e3
    kk = np.zeros((N, dh))
    kk[4, 0] = 1.0
    assert np.allclose(dit.attention_rows(q, kk, v), v[4:5], atol=1e-12)
    # permuting keys and values together changes nothing
    q = rng.normal(size=(4, dh))
    perm = rng.permutation(N)
    assert np.allclose(dit.attention_rows(q, k, v), dit.attention_rows(q, k[perm], v[perm]), atol=1e-13)
    # two keys: a logistic mix with weight sigmoid((q.k0 - q.k1)/sqrt(d))
    q1 = rng.normal(size=(1, dh))
    a = scipy.special.expit(((q1 @ k[0]) - (q1 @ k[1]))[0] / math.sqrt(dh))
    assert np.allclose(dit.attention_rows(q1, k[:2], v[:2]), a * v[0] + (1 - a) * v[1], atol=1e-13)


def test_attention_heads_are_independent_column_slices():
    N, heads, dh = 11, 3, 4
    q, k, v = (rng.normal(size=(N, heads * dh)) for _ in range(3))
    o = dit.attention(q, k, v, heads, chunk=4)
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        assert np.allclose(o[:, sl], dit.attention_rows(q[:, sl], k[:, sl], v[:, sl]), atol=1e-13)


def test_patchify_layout_and_roundtrip():
    C, T, H, W, p = 3, 2, 4, 6, 2
    x = rng.normal(size=(C, T, H, W))
    tok = dit.patchify(x, p)
    Hp, Wp = H // p, W // p
    for t in range(T):
        for i in range(Hp):
            for j in range(Wp):
                for c in range(C):
                    for a in range(p):
                        for b in range(p):
                            assert tok[(t * Hp + i) * Wp + j, c * p * p + a * p + b] == x[c, t, p * i + a, p * j + b]
    assert np.array_equal(dit.unpatchify(tok, x.shape, p), x)


def test_euler_closed_forms():
    K = 10
    sig = I.sigmas(K)
    assert sig[0] == 1.0 and sig[-1] == 0.0
    x = rng.normal(size=(5,))
    v = rng.normal(size=(5,))
    y = x.copy()
    for k in range(K):
        y = dit.euler(y, v, sig[k], sig[k + 1])
    assert np.allclose(y, x - v, atol=1e-14)          # sum of steps = sigma_{K+1} - sigma_1 = -1
    assert np.array_equal(dit.euler(x, np.zeros(5), sig[0], sig[1]), x)


def _tiny():
    w = I.WORKLOADS["dit-tiny-f32"]
    return w, I.Weights(w.model, w.cfg_id)


def test_block_with_zero_output_projections_is_identity():
    w, _ = _tiny()
    W = I.Weights(w.model, w.cfg_id, zero_out=("w_o", "b_o", "w_2", "b_2"))
    P = dit.Params(W)
    mods, _ = dit.step_modulation(P, 0.7)
    h = I.hidden_state(w.model, (1,)).astype(np.float64)
    assert np.array_equal(dit.block(P, 0, mods[0], h), h)


def test_block_with_zero_gates_is_identity_and_gates_are_linear():
    w, W = _tiny()
    P = dit.Params(W)
    mods, _ = dit.step_modulation(P, 0.3)
    h = I.hidden_state(w.model, (2,)).astype(np.float64)
    m = mods[0].copy()
    m[2] = 0.0
    m[5] = 0.0
    assert np.array_equal(dit.block(P, 0, m, h), h)
    # with the MLP gate closed, the attention update is linear in gate1
    m2 = m.copy()
    m2[2] = 1.0
    m3 = m.copy()
    m3[2] = 2.0
    d2 = dit.block(P, 0, m2, h) - h
    d3 = dit.block(P, 0, m3, h) - h
    assert np.allclose(d3, 2 * d2, rtol=1e-12, atol=1e-15)


def test_sampled_rows_match_full_block():
    w, W = _tiny()
    P = dit.Params(W)
    mods, _ = dit.step_modulation(P, 0.5)
    h = I.hidden_state(w.model, (3,)).astype(np.float64)
    full = dit.block(P, 1, mods[1], h)
    rows = np.array([0, 5, 100, 255, 256, 271])
    assert np.allclose(dit.block(P, 1, mods[1], h, rows=rows), full[rows], rtol=1e-12, atol=1e-14)


def test_head_modulation_uses_time_embedding():
    w, W = _tiny()
    P = dit.Params(W)
    _, hm = dit.step_modulation(P, 0.25)
    c = dit.time_embedding(P, 0.25)
    assert np.allclose(hm - W.get("head_mod").astype(np.float64), np.stack([c, c]), atol=1e-15)


def test_bf16_rounding_is_ties_to_even():
    a = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5], np.float32)
    r = I.round_bf16(a)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1.0)
    assert list(r) == [1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5]
    import torch
    x = np.random.default_rng(0).normal(size=4096).astype(np.float32)
    assert np.array_equal(I.round_bf16(x), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


class _Stub:
    """Hand-built weights for special-case pins."""

    def __init__(self, m, blocks):
        self.m = m
        self._b = blocks

    def block(self, l, name):
        return self._b[name]

    def get(self, name):  # pragma: no cover - not used by block()
        raise KeyError(name)


def _stub_model():
    return I.ModelShape(1, 8, 2, 4, 32, 16, 1, 2, 2, 2, 0, "f32")


def test_block_attention_special_case_is_mean_of_values():
    # W_q = 0 makes every query zero: attention averages the value rows, so with
    # W_o = I, b_o = 0, gate1 = 1 and the MLP gate closed the block adds
    # mean_n(LN-mod(h)_n W_v^T + b_v) to every row
    m = _stub_model()
    d, F = m.hidden, m.mlp_hidden
    Wv = rng.normal(size=(d, d))
    bv = rng.normal(size=d)
    blocks = {"w_qkv": np.concatenate([np.zeros((d, d)), rng.normal(size=(d, d)), Wv]),
              "b_qkv": np.concatenate([np.zeros(d), rng.normal(size=d), bv]),
              "w_o": np.eye(d), "b_o": np.zeros(d),
              "w_1": rng.normal(size=(F, d)), "b_1": rng.normal(size=F),
              "w_2": rng.normal(size=(d, F)), "b_2": rng.normal(size=d)}
    P = dit.Params(_Stub(m, blocks))
    h = rng.normal(size=(5, d))
    shift, scale = rng.normal(size=d), rng.normal(size=d)
    mod = np.stack([shift, scale, np.ones(d), np.zeros(d), np.zeros(d), np.zeros(d)])
    a = (h - h.mean(1, keepdims=True)) / np.sqrt(h.var(1, keepdims=True) + m.ln_eps) * (1 + scale) + shift
    expect = h + (a @ Wv.T + bv).mean(axis=0)
    assert np.allclose(dit.block(P, 0, mod, h), expect, rtol=1e-12, atol=1e-12)


def test_block_mlp_special_case_is_gated_gelu():
    # attention gate closed; W_1 = [I; 0], W_2 = [I, 0], zero biases: the block adds
    # gate2 * GELU(LN-mod2(h)) -- the activation sits between the two projections
    m = _stub_model()
    d, F = m.hidden, m.mlp_hidden
    w1 = np.zeros((F, d))
    w1[:d] = np.eye(d)
    w2 = np.zeros((d, F))
    w2[:, :d] = np.eye(d)
    blocks = {"w_qkv": rng.normal(size=(3 * d, d)), "b_qkv": rng.normal(size=3 * d),
              "w_o": rng.normal(size=(d, d)), "b_o": rng.normal(size=d),
              "w_1": w1, "b_1": np.zeros(F), "w_2": w2, "b_2": np.zeros(d)}
    P = dit.Params(_Stub(m, blocks))
    h = rng.normal(size=(4, d))
    shift2, scale2, gate2 = rng.normal(size=d), rng.normal(size=d), rng.normal(size=d)
    mod = np.stack([np.zeros(d), np.zeros(d), np.zeros(d), shift2, scale2, gate2])
    a2 = (h - h.mean(1, keepdims=True)) / np.sqrt(h.var(1, keepdims=True) + m.ln_eps) * (1 + scale2) + shift2
    z = a2 * 0.5 * (1 + scipy.special.erf(a2 / np.sqrt(2)))          # erf-GELU, within 2e-3
    got = dit.block(P, 0, mod, h) - h
    assert np.allclose(got, gate2 * z, atol=3e-3 * np.abs(gate2).max())
    assert not np.allclose(got, gate2 * a2, atol=1e-3)


class _StubAll(_Stub):
    def __init__(self, m, glob, blocks):
        super().__init__(m, None)
        self._g = glob
        self._bl = blocks

    def block(self, l, name):
        return self._bl[l][name]

    def get(self, name):
        return self._g[name]


def test_time_embedding_and_modulation_closed_form():
    """Hand-built conditioning weights that reduce the timestep MLP and the shared
    modulation projection to per-element closed forms, evaluated with scalar math:
    W_t1 picks one sinusoid per hidden unit (a cosine for most, a scaled sine for the
    last), W_t2 is diagonal plus one off-diagonal entry, W_m stacks +I, -3I, zero and a diagonal.  A dropped
    SiLU, a SiLU in the wrong place, a transposed weight, a wrong [6, d] row order or
    a missing [c; c] head offset each changes the result."""
    m = I.ModelShape(2, 8, 2, 4, 32, 16, 1, 2, 2, 2, 0, "f32")
    d, nf = m.hidden, m.t_freq
    half = nf // 2
    r = np.random.default_rng(5)
    w_t1 = np.zeros((d, nf))
    pick = [3 * i for i in range(d - 1)]
    for i, f in enumerate(pick):
        w_t1[i, f] = 1.0
    w_t1[d - 1, half + 5] = -2.0                      # the sine of frequency 5
    b_t1 = 0.1 * np.arange(d) - 0.3
    diag_t2 = 0.5 * (np.arange(d) + 1)
    b_t2 = 0.01 * np.arange(d)
    w_m = np.zeros((6 * d, d))
    w_m[0:d] = np.eye(d)
    w_m[d:2 * d] = -3.0 * np.eye(d)
    diag_m5 = r.normal(size=d)
    w_m[5 * d:6 * d] = np.diag(diag_m5)
    b_m = r.normal(size=6 * d)
    head_mod = r.normal(size=(2, d))
    offs = [r.normal(size=(6, d)) for _ in range(m.n_blocks)]
    w_t2 = np.diag(diag_t2)
    w_t2[0, d - 1] = 0.7                              # one off-diagonal entry: orientation matters
    glob = {"w_t1": w_t1, "b_t1": b_t1, "w_t2": w_t2, "b_t2": b_t2,
            "w_m": w_m, "b_m": b_m, "head_mod": head_mod}
    P = dit.Params(_StubAll(m, glob, [{"mod_offset": o} for o in offs]))

    def silu(z):
        return z / (1.0 + math.exp(-z))

    for sigma in (0.0, 0.37, 1.0):
        t = 1000.0 * sigma
        freq = [10000.0 ** (-i / half) for i in range(half)]
        pre = [math.cos(t * freq[f]) + b_t1[i] for i, f in enumerate(pick)]
        pre.append(-2.0 * math.sin(t * freq[5]) + b_t1[d - 1])
        c = np.array([diag_t2[i] * silu(pre[i]) + b_t2[i] for i in range(d)])
        c[0] += 0.7 * silu(pre[d - 1])
        s = np.array([silu(ci) for ci in c])
        mm = b_m.reshape(6, d).copy()
        mm[0] += s
        mm[1] += -3.0 * s
        mm[5] += diag_m5 * s
        assert np.allclose(dit.time_embedding(P, sigma), c, rtol=1e-13, atol=1e-14)
        blocks, head = dit.step_modulation(P, sigma)
        for l in range(m.n_blocks):
            assert np.allclose(blocks[l], mm + offs[l], rtol=1e-13, atol=1e-14)
        assert np.allclose(head, head_mod + np.stack([c, c]), rtol=1e-13, atol=1e-14)
    # at t = 0 every cosine feature is 1 and every sine 0 (closed form of the features)
    blocks0, _ = dit.step_modulation(P, 0.0)
    z = 1.0 + b_t1[0]
    zl = b_t1[d - 1]
    c0 = diag_t2[0] * z / (1.0 + math.exp(-z)) + 0.7 * zl / (1.0 + math.exp(-zl)) + b_t2[0]
    assert blocks0[0][0, 0] == pytest.approx(c0 / (1.0 + math.exp(-c0)) + b_m[0] + offs[0][0, 0], rel=1e-14)
