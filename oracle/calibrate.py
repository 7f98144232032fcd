"""Anchor calibration of the run tables (Sec. 3.1 after Eq. 4; Eq. 5-7), float64.

Test infrastructure only (see oracle/__init__.py).

For one anchor clip, a full denoising trace stores (x_k, u_k, r_k) for every step
k (x_k is the latent the step starts from, u_k block 0's modulated input of the
video rows, r_k = h_out - h_in over the video rows).  For a run that refreshes at
step j and reuses r_j for h steps:

  * Eq. 5, the anchor input drift at the l-th reuse:
        d_{j,l} = ||u_{j+l} - u_j||_2 / (||u_{j+l}||_2 + eps);
  * Eq. 6, the signed output perturbation against the full trace:
        e_{j,l} = H_{j+l}(x_{j+l}, r_j) - H_{j+l}(x_{j+l}, r_{j+l}),
    H_k(x, r) being the denoiser output the head gives for g = h_in(x)[video] + r;
  * Eq. 7, the joint run response:
        G_{j,h} = sum_{l=1..h} P_{j+l} e_{j,l},   q_{j,h} = ||G_{j,h}||_2 / (||x_K||_2 + eps),
    P_t the Jacobian of the terminal latent with respect to the denoiser output
    of step t along the frozen full trace.

P_t e is a Jacobian-vector product through the frozen sampler tail: the Euler
update of step t adds (sigma_{t+1} - sigma_t) e to x_{t+1}, and every later step
k carries the tangent as dx_{k+1} = dx_k + (sigma_{k+1} - sigma_k) J_k dx_k with
J_k the Jacobian of the full network at x_k.  The tangent of the network is
written out layer by layer (LayerNorm with modulation, the projections,
softmax attention, GELU-tanh, the gated residuals, patch embedding and head);
the modulation depends on the noise level only, so it carries no tangent.

Readings where the paper is silent:
  * "terminal latent x_K" is the sampler's output after the last step (x_{K+1}
    in the 1-based step numbering used here);
  * the tables cover runs with j + h <= K; entries of runs that would pass the
    last step are 0 (the schedule never prices them);
  * the norms are over the whole tensor of one clip.
"""
from __future__ import annotations

import math

import numpy as np

from . import dit

F = np.float64


# ----------------------------------------------------------------------------
# tangents of the network's pieces
# ----------------------------------------------------------------------------
def jvp_layer_norm(x, dx, eps):
    """y = (x - mu) r with r = (var + eps)^-1/2: dr = -r^3 mean((x - mu) dx), so
    dy = r [dxc - y mean(y dxc)], dxc = dx - mean(dx)."""
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(var + eps)
    y = xc * r
    dxc = dx - dx.mean(axis=-1, keepdims=True)
    dy = r * (dxc - y * (y * dxc).mean(axis=-1, keepdims=True))
    return y, dy


def jvp_modulate(x, dx, shift, scale, eps):
    y, dy = jvp_layer_norm(x, dx, eps)
    return y * (1.0 + scale) + shift, dy * (1.0 + scale)


def jvp_gelu_tanh(z, dz):
    c = math.sqrt(2.0 / math.pi)
    u = c * (z + 0.044715 * z * z * z)
    t = np.tanh(u)
    g = 0.5 * z * (1.0 + t)
    dg = (0.5 * (1.0 + t) + 0.5 * z * (1.0 - t * t) * c * (1.0 + 3.0 * 0.044715 * z * z)) * dz
    return g, dg


def jvp_attention(q, k, v, dq, dk, dv, heads):
    """O = softmax(q k^T / sqrt(d_h)) v per head: dS = (dq k^T + q dk^T) / sqrt(d_h),
    dP = P (dS - rowsum(P dS)), dO = dP v + P dv."""
    r, d = q.shape
    dh = d // heads
    out = np.empty((r, d), F)
    dout = np.empty((r, d), F)
    for hd in range(heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        qs, ks, vs = q[:, sl], k[:, sl], v[:, sl]
        s = (qs @ ks.T) / math.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        ds = (dq[:, sl] @ ks.T + qs @ dk[:, sl].T) / math.sqrt(dh)
        dp = p * (ds - (p * ds).sum(axis=1, keepdims=True))
        out[:, sl] = p @ vs
        dout[:, sl] = dp @ vs + p @ dv[:, sl]
    return out, dout


def jvp_block(P, l, mod6, h, dh):
    m = P.m
    d = m.hidden
    eps = m.ln_eps
    shift1, scale1, gate1, shift2, scale2, gate2 = mod6
    a, da = jvp_modulate(h, dh, shift1, scale1, eps)
    wq, bq = P.b(l, "w_qkv"), P.b(l, "b_qkv")
    qkv = a @ wq.T + bq
    dqkv = da @ wq.T
    o, do = jvp_attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:],
                          dqkv[:, :d], dqkv[:, d:2 * d], dqkv[:, 2 * d:], m.heads)
    wo = P.b(l, "w_o")
    h1 = h + gate1 * (o @ wo.T + P.b(l, "b_o"))
    dh1 = dh + gate1 * (do @ wo.T)
    a2, da2 = jvp_modulate(h1, dh1, shift2, scale2, eps)
    w1, w2 = P.b(l, "w_1"), P.b(l, "w_2")
    z, dz = jvp_gelu_tanh(a2 @ w1.T + P.b(l, "b_1"), da2 @ w1.T)
    h2 = h1 + gate2 * (z @ w2.T + P.b(l, "b_2"))
    dh2 = dh1 + gate2 * (dz @ w2.T)
    return h2, dh2


def jvp_network(P, sigma, x, dx, txt):
    """The full network of the step at noise level sigma (the refresh path: patch
    embedding, block stack, head on h_out): v = F(x) and dv = J dx."""
    m = P.m
    mods, head_mod = dit.step_modulation(P, sigma)
    h = dit.embed(P, x, txt)
    dpv = dit.patchify(dx.astype(F), m.patch) @ P.g("w_pe").T       # text rows carry no tangent
    dh = np.concatenate([dpv, np.zeros((m.n_txt, m.hidden), F)], axis=0)
    for l in range(m.n_blocks):
        h, dh = jvp_block(P, l, mods[l], h, dh)
    y, dy = jvp_modulate(h[: m.n_v], dh[: m.n_v], head_mod[0], head_mod[1], m.ln_eps)
    wh = P.g("w_head")
    v = dit.unpatchify(y @ wh.T + P.g("b_head"), m.latent_shape, m.patch)
    dv = dit.unpatchify(dy @ wh.T, m.latent_shape, m.patch)
    return v, dv


# ----------------------------------------------------------------------------
# anchor trace and the tables
# ----------------------------------------------------------------------------
class Trace:
    """Full (uncached) trace of one anchor clip: x[k], u[k], r[k], v[k] for steps
    k = 1..K (index k - 1), and the terminal latent x_out."""

    def __init__(self, P, x1, txt, sigmas):
        m = P.m
        self.P, self.txt, self.sigmas = P, txt, np.asarray(sigmas, F)
        K = len(sigmas) - 1
        self.K = K
        self.x, self.u, self.r, self.v = [], [], [], []
        x = x1.astype(F)
        for k in range(1, K + 1):
            mods, head_mod = dit.step_modulation(P, sigmas[k - 1])
            h_in = dit.embed(P, x, txt)
            h_out = dit.backbone(P, mods, h_in)
            v = dit.head(P, head_mod, h_out[: m.n_v])
            self.x.append(x)
            self.u.append(dit.backbone_input(P, h_in, mods[0]))
            self.r.append(h_out[: m.n_v] - h_in[: m.n_v])
            self.v.append(v)
            x = dit.euler(x, v, sigmas[k - 1], sigmas[k])
        self.x_out = x


def interface(P, sigma, x, txt, r):
    """H_k(x, r): the denoiser output for g = h_in(x)[video] + r at noise level sigma."""
    _, head_mod = dit.step_modulation(P, sigma)
    g = dit.embed(P, x, txt)[: P.m.n_v] + r
    return dit.head(P, head_mod, g)


def input_drift(tr: Trace, j, ell, eps):
    """Eq. 5 (1-based steps)."""
    du = tr.u[j + ell - 1] - tr.u[j - 1]
    return float(np.linalg.norm(du)) / (float(np.linalg.norm(tr.u[j + ell - 1])) + eps)


def output_perturbation(tr: Trace, j, ell):
    """Eq. 6 (1-based steps)."""
    k = j + ell
    s = tr.sigmas[k - 1]
    return (interface(tr.P, s, tr.x[k - 1], tr.txt, tr.r[j - 1])
            - interface(tr.P, s, tr.x[k - 1], tr.txt, tr.r[k - 1]))


def tail_jvp(tr: Trace, t, e):
    """P_t e: the terminal-latent tangent when the denoiser output of step t moves by e."""
    sig = tr.sigmas
    dx = (sig[t] - sig[t - 1]) * e
    for k in range(t + 1, tr.K + 1):
        _, dv = jvp_network(tr.P, sig[k - 1], tr.x[k - 1], dx, tr.txt)
        dx = dx + (sig[k] - sig[k - 1]) * dv
    return dx


def tail_rerun(tr: Trace, t, e):
    """The terminal latent when the denoiser output of step t is v_t + e and every later
    step runs the full network (the finite-difference counterpart of tail_jvp)."""
    P, sig = tr.P, tr.sigmas
    x = tr.x[t - 1] + (sig[t] - sig[t - 1]) * (tr.v[t - 1] + e)
    for k in range(t + 1, tr.K + 1):
        mods, head_mod = dit.step_modulation(P, sig[k - 1])
        h_in = dit.embed(P, x, tr.txt)
        h_out = dit.backbone(P, mods, h_in)
        x = dit.euler(x, dit.head(P, head_mod, h_out[: P.m.n_v]), sig[k - 1], sig[k])
    return x


def run_tables(tr: Trace, h_max, eps):
    """(q, d) [(K-1), h_max]: row j - 1 = refresh step j, column h - 1 = run length h
    (Eq. 5, Eq. 7); runs with j + h > K are 0."""
    K = tr.K
    q = np.zeros((K - 1, h_max), F)
    d = np.zeros((K - 1, h_max), F)
    xn = float(np.linalg.norm(tr.x_out))
    for j in range(1, K):
        G = np.zeros_like(tr.x_out)
        for h in range(1, h_max + 1):
            if j + h > K:
                break
            G = G + tail_jvp(tr, j + h, output_perturbation(tr, j, h))
            q[j - 1, h - 1] = float(np.linalg.norm(G)) / (xn + eps)
            d[j - 1, h - 1] = input_drift(tr, j, h, eps)
    return q, d
