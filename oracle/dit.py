"""Spatiotemporal video DiT, its cache boundary and the Euler sampler, in float64.

Test infrastructure only (see oracle/__init__.py).

The paper treats the generator as frozen and names only its interface (Eq. 1):
r_k = F_k(u_k), eps_k = H_k(x_k, r_k).  The generator below is a stand-in with
the structure of the paper's video DiTs (joint video+text self-attention,
AdaLN modulation from the timestep, flow-matching Euler sampling); every
architectural detail is a reading, listed here:

  * timestep t = 1000 sigma; features [cos(t w_i), sin(t w_i)], w_i = 10000^(-i/128);
    c = W_t2 SiLU(W_t1 e + b_t1) + b_t2; shared modulation m = W_m SiLU(c) + b_m
    ([6, d]); block l uses m + M_l = (shift1, scale1, gate1, shift2, scale2, gate2);
    the head uses (shift_f, scale_f) = M_f + [c; c]
  * patchify: token n = (t Hp + i) Wp + j; patch-vector index c p^2 + a p + b holds
    x[c, t, p i + a, p j + b];  h_in = patch W_pe^T + b_pe + pos for video rows,
    the text embeddings for the rows after them
  * block: a = LN(h)(1 + scale1) + shift1; [Q|K|V] = a W_qkv^T + b_qkv (column
    s d + head d_h + i); O = softmax(Q K^T / sqrt(d_h)) V per head over all rows;
    h += gate1 (O W_o^T + b_o); a2 = LN(h)(1 + scale2) + shift2;
    h += gate2 (GELU_tanh(a2 W_1^T + b_1) W_2^T + b_2).  LN: biased variance, no affine.
  * head: y = LN(g)(1 + scale_f) + shift_f; v = unpatchify(y W_head^T + b_head)
  * sampler: x_{k+1} = x_k + (sigma_{k+1} - sigma_k) v_k
  * cache boundary: F_k is the block stack; r_k = h_out - h_in over the video
    rows; H_k(x_k, r) = head(h_in(x_k)[video] + r) followed by the Euler update;
    the backbone input u_k is block 0's modulated input over the video rows.
    A refresh step feeds the head h_out itself (not h_in + r).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from threadpoolctl import threadpool_limits

F = np.float64


def _workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _by_rows(fn, x, *args, min_rows=4096):
    """fn(x, *args) for a row-wise fn (each output row depends on its input row only),
    evaluated on row ranges in worker threads; the values are those of one call."""
    n = x.shape[0]
    nw = _workers()
    if n < min_rows or nw == 1:
        return fn(x, *args)
    bounds = np.linspace(0, n, nw + 1).astype(int)
    out = np.empty(x.shape, F)

    def run(i):
        out[bounds[i]: bounds[i + 1]] = fn(x[bounds[i]: bounds[i + 1]], *args)

    with ThreadPoolExecutor(nw) as ex:
        list(ex.map(run, range(nw)))
    return out


def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(z):
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z * z * z)))


def layer_norm(x, eps):
    """Per-row normalisation over the last axis, biased variance, no affine."""
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    return xc / np.sqrt(var + eps)


def modulate(x, shift, scale, eps):
    return layer_norm(x, eps) * (1.0 + scale) + shift


def timestep_features(t, n_freq=256):
    half = n_freq // 2
    i = np.arange(half, dtype=F)
    w = np.power(10000.0, -i / half)
    arg = F(t) * w
    return np.concatenate([np.cos(arg), np.sin(arg)])


class Params:
    """float64 views of a `Weights` object (lazy per block)."""

    def __init__(self, W):
        self.W = W
        self.m = W.m
        self._c = {}

    def g(self, name):
        if name not in self._c:
            self._c[name] = self.W.get(name).astype(F)
        return self._c[name]

    def b(self, l, name):
        key = (l, name)
        if key not in self._c:
            self._c[key] = self.W.block(l, name).astype(F)
        return self._c[key]


def time_embedding(P: Params, sigma):
    e = timestep_features(1000.0 * F(sigma), P.m.t_freq)
    hdn = silu(P.g("w_t1") @ e + P.g("b_t1"))
    return P.g("w_t2") @ hdn + P.g("b_t2")


def step_modulation(P: Params, sigma):
    """Per-block [6, d] modulation for every block, and the head's (shift_f, scale_f)."""
    c = time_embedding(P, sigma)
    d = P.m.hidden
    m = (P.g("w_m") @ silu(c) + P.g("b_m")).reshape(6, d)
    blocks = [m + P.b(l, "mod_offset") for l in range(P.m.n_blocks)]
    head = P.g("head_mod") + np.stack([c, c])
    return blocks, head


# ----------------------------------------------------------------------------
# patchify / embed / head
# ----------------------------------------------------------------------------
def patchify(x, p):
    """[C, T, H, W] -> [T*Hp*Wp, C*p*p]."""
    C, T, H, W = x.shape
    Hp, Wp = H // p, W // p
    y = x.reshape(C, T, Hp, p, Wp, p)               # c, t, i, a, j, b
    y = y.transpose(1, 2, 4, 0, 3, 5)               # t, i, j, c, a, b
    return y.reshape(T * Hp * Wp, C * p * p)


def unpatchify(tok, shape, p):
    C, T, H, W = shape
    Hp, Wp = H // p, W // p
    y = tok.reshape(T, Hp, Wp, C, p, p).transpose(3, 0, 1, 4, 2, 5)   # c, t, i, a, j, b
    return y.reshape(C, T, H, W)


def embed(P: Params, x, txt):
    """Backbone input h_in [N, d]: patch embedding + position for video rows, then text."""
    pv = patchify(x.astype(F), P.m.patch)
    hv = pv @ P.g("w_pe").T + P.g("b_pe") + P.g("pos")
    return np.concatenate([hv, txt.astype(F)], axis=0)


def backbone_input(P: Params, h_in, mod0):
    """u_k: block 0's modulated input over the video rows."""
    return modulate(h_in[: P.m.n_v], mod0[0], mod0[1], P.m.ln_eps)


def head(P: Params, head_mod, g):
    y = modulate(g, head_mod[0], head_mod[1], P.m.ln_eps)
    tok = y @ P.g("w_head").T + P.g("b_head")
    return unpatchify(tok, P.m.latent_shape, P.m.patch)


def euler(x, v, s0, s1):
    return x + (F(s1) - F(s0)) * v


# ----------------------------------------------------------------------------
# attention and the transformer block
# ----------------------------------------------------------------------------
def attention_rows(q, k, v):
    """softmax(q k^T / sqrt(d_h)) v for one head; q [r, d_h], k, v [N, d_h]."""
    return _softmax_times_v(q @ k.T, v, q.shape[1])


def _softmax_times_v(s, v, dh):
    """softmax(s / sqrt(d_h)) v for scores s = q k^T.  The steps run in place in s
    (the same operations in the same order as with fresh arrays, so the same values;
    large fresh arrays cost page faults that serialise the worker threads)."""
    s /= math.sqrt(dh)
    s -= s.max(axis=1, keepdims=True)
    np.exp(s, out=s)
    s /= s.sum(axis=1, keepdims=True)
    return s @ v


def split_heads(k, v, heads):
    """Per head: (k_h^T, v_h) as contiguous arrays [d_h, N] and [N, d_h].  The same
    values as the column slices of k and v; the products read them faster."""
    dh = k.shape[1] // heads
    return [(np.ascontiguousarray(k[:, h * dh:(h + 1) * dh].T), np.ascontiguousarray(v[:, h * dh:(h + 1) * dh]))
            for h in range(heads)]


def attention(q, k, v, heads, chunk=2048, kv_heads=None):
    """Multi-head attention over all rows; q [r, d], k, v [N, d] (heads concatenated).
    Query rows are processed in chunks only to bound memory (rows are independent).
    kv_heads (optional): split_heads(k, v, heads), which replaces k and v."""
    r, d = q.shape
    dh = d // heads
    out = np.empty((r, d), F)
    for hd in range(heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        kt, vh = (k[:, sl].T, v[:, sl]) if kv_heads is None else kv_heads[hd]
        for a in range(0, r, chunk):
            out[a: a + chunk, sl] = _softmax_times_v(q[a: a + chunk, sl] @ kt, vh, dh)
    return out


def _block_rows(P: Params, l, mod6, h, a, kv_heads):
    """The part of block l after the keys and values: rows h, with modulated input a,
    attend to every row's keys and values (kv_heads = split_heads(k, v)); each output
    row depends on its own row only."""
    d = P.m.hidden
    eps = P.m.ln_eps
    _, _, gate1, shift2, scale2, gate2 = mod6
    wq, bq = P.b(l, "w_qkv"), P.b(l, "b_qkv")
    q = a @ wq[:d].T + bq[:d]
    o = attention(q, None, None, P.m.heads, chunk=64, kv_heads=kv_heads)
    hr = h + gate1 * (o @ P.b(l, "w_o").T + P.b(l, "b_o"))
    a2 = modulate(hr, shift2, scale2, eps)
    z = gelu_tanh(a2 @ P.b(l, "w_1").T + P.b(l, "b_1"))
    return hr + gate2 * (z @ P.b(l, "w_2").T + P.b(l, "b_2"))


def block(P: Params, l, mod6, h, rows=None, chunk=256):
    """One transformer block on h [N, d]; returns the updated rows (all rows, or
    only `rows` -- every row's keys and values are still used).
    Given the keys and values, rows are independent: they are evaluated in chunks
    of `chunk` rows in worker threads (one BLAS thread each), only to use the
    host's cores with cache-sized temporaries."""
    d = P.m.hidden
    shift1, scale1 = mod6[0], mod6[1]
    a = _by_rows(modulate, h, shift1, scale1, P.m.ln_eps)
    wq, bq = P.b(l, "w_qkv"), P.b(l, "b_qkv")
    kv = a @ wq[d:].T + bq[d:]                 # keys and values of every row
    kv_heads = split_heads(kv[:, :d], kv[:, d:], P.m.heads)
    del kv
    sel = np.arange(h.shape[0]) if rows is None else np.arange(h.shape[0])[rows]
    out = np.empty((len(sel), d), F)
    starts = range(0, len(sel), chunk)

    def run(s):
        rr = sel[s: s + chunk]
        out[s: s + chunk] = _block_rows(P, l, mod6, h[rr], a[rr], kv_heads)

    for name in ("w_o", "b_o", "w_1", "b_1", "w_2", "b_2"):
        P.b(l, name)                           # load once, before the threads share P
    with threadpool_limits(1), ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(run, starts))
    return out


def backbone(P: Params, mods, h_in, memo=None):
    """F: the whole block stack on h_in [N, d]; returns h_out.
    memo (optional, for long runs that may be interrupted): an object whose
    load(l, h) returns block l's output for the input h if it holds it (else None)
    and whose save(l, h, out) records it; the values are those of block() itself."""
    h = h_in
    for l in range(P.m.n_blocks):
        out = memo.load(l, h) if memo is not None else None
        if out is None:
            out = block(P, l, mods[l], h)
            if memo is not None:
                memo.save(l, h, out)
        h = out
    return h
