"""Edge shapes of the device path against the oracle, through the C ABI.

Small seeded models whose token counts leave ragged tails everywhere: fewer
tokens than one attention tile (37, head_dim 72), fewer than one MFMA row tile
and no text (16), one partial GEMM row tile (111), several row tiles, attention
tiles and query blocks with a ragged last one (328), the fp32 path at a
ragged count (95), and 3,597 tokens x 30 heads, where the attention's query
blocks outnumber the resident workgroups by just over three rounds on MI355X, so
the last partial round runs as split key halves merged by the combine kernel.
The fused head's extremes: one video token (one partial token tile) at d = 256
(one 32-wide chunk per wave) and d = 2048 (eight chunks per wave).
Also: empty index lists leave every buffer untouched."""
import numpy as np
import pytest

from oracle import dit, runtime
from paper_2608_16354_amd import inputs as I
from tests.gpu_util import mod_input, rel_l2, say, t
from tests.test_gpu_kernels import _Head, _OneBlock, _head_tol

pytestmark = pytest.mark.gpu


def _shape(d, heads, hd, f, lat, n_txt, dtype):
    return I.ModelShape(n_blocks=1, hidden=d, heads=heads, head_dim=hd, mlp_hidden=f, lat_c=16,
                        lat_t=lat[0], lat_h=lat[1], lat_w=lat[2], patch=2, n_txt=n_txt, dtype=dtype)


EDGE = {
    "bf16-N37-hd72": (_shape(1152, 16, 72, 4608, (2, 6, 10), 7, "bf16"), 91),
    "bf16-N16-notext": (_shape(256, 4, 64, 1024, (1, 8, 8), 0, "bf16"), 92),
    "bf16-N111": (_shape(256, 4, 64, 1024, (3, 10, 12), 21, "bf16"), 93),
    "bf16-N328": (_shape(384, 6, 64, 1536, (5, 14, 18), 13, "bf16"), 94),
    "f32-N95": (_shape(256, 4, 64, 1024, (3, 10, 12), 5, "f32"), 95),
    "bf16-N3597-h30-split": (_shape(1920, 30, 64, 7680, (10, 32, 44), 77, "bf16"), 96),
    "bf16-N1-d256": (_shape(256, 4, 64, 1024, (1, 2, 2), 3, "bf16"), 97),
    "bf16-N40-d2048": (_shape(2048, 32, 64, 8192, (2, 8, 10), 5, "bf16"), 98),
}


@pytest.fixture(scope="module")
def api():
    from paper_2608_16354_amd import api as A
    A.L.load()
    return A


def _bf(m):
    return m.dtype == "bf16"


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_block_forward(api, dev, name):
    import torch
    m, cid = EDGE[name]
    W = I.Weights(m, cid)
    dm = api.DeviceModel(_OneBlock(W, 0), dev)
    ws = api.Workspace(m, 1, dev)
    h = I.hidden_state(m, (40,))
    mod = mod_input(m, (41,))
    dh = t(h[None], dev)
    say("edge block_forward", name, "N =", m.n_tok)
    api.dc_block_forward(dm, 0, t(mod, dev), dh, [0], ws)
    torch.cuda.synchronize()
    got = dh[0].cpu().numpy()
    want = dit.block(dit.Params(W), 0, mod.astype(np.float64), h.astype(np.float64))
    err_h, err_d = rel_l2(got, want), rel_l2(got - h, want - h)
    say(name, "block rel-L2 h_out", err_h, "update", err_d)
    if _bf(m):
        assert err_h < 1e-2 and err_d < 2e-2
    else:
        assert err_h < 1e-5 and err_d < 1e-5


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_patch_embed_and_head(api, dev, name):
    import torch
    m, cid = EDGE[name]
    W = I.Weights(m, cid)
    P = dit.Params(W)
    dm = api.DeviceModel(_Head(W), dev)
    ws = api.Workspace(m, 1, dev)
    x = I.latent(m, cid, 0)
    txt = I.text(m, cid, 0)
    h_in = torch.zeros((1, m.n_tok, m.hidden), device=dev)
    say("edge patch_embed", name, "N_v =", m.n_v)
    api.dc_patch_embed(dm, t(x[None], dev), t(txt[None], dev), h_in, [0], ws)
    torch.cuda.synchronize()
    got = h_in[0].cpu().numpy()
    want = dit.embed(P, x.astype(np.float64), txt)
    assert rel_l2(got[: m.n_v], want[: m.n_v]) < (1e-5 if _bf(m) else 1e-6)
    assert np.array_equal(got[m.n_v:], txt)
    g = I.hidden_state(m, (42,))
    hm = mod_input(m, (43,))[:2]
    dx = t(x[None], dev)
    say("edge head_euler", name)
    api.dc_head_euler(dm, t(hm, dev), t(g[None], dev), dx, -0.02, [0], ws)
    torch.cuda.synchronize()
    v = dit.head(P, hm.astype(np.float64), g[: m.n_v].astype(np.float64))
    want_x = dit.euler(x.astype(np.float64), v, 0.52, 0.5)
    err = rel_l2(dx[0].cpu().numpy() - x, want_x - x)
    say(name, "head update rel-L2", err)
    assert err < _head_tol(m)


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_drift_and_cache(api, dev, name):
    import torch
    m, cid = EDGE[name]
    cfg = api.model_cfg(m)
    ws = api.Workspace(m, 1, dev)
    mdt = torch.bfloat16 if _bf(m) else torch.float32
    h_in = I.hidden_state(m, (44,))
    mod0 = mod_input(m, (45,))[:2]
    ref = I.normal((m.n_v, m.hidden), 1.0, (46,))
    ref = I.round_bf16(ref) if _bf(m) else ref
    u_ref = t(ref[None], dev, mdt)
    sums = torch.zeros((1, 4), dtype=torch.float64, device=dev)
    say("edge drift", name)
    api.dc_drift_l1(cfg, t(h_in[None], dev), t(mod0, dev), u_ref, 0, sums, [0], ws)
    torch.cuda.synchronize()
    u = dit.modulate(h_in[: m.n_v].astype(np.float64), mod0[0].astype(np.float64),
                     mod0[1].astype(np.float64), m.ln_eps)
    want = runtime.drift_sums(u, ref.astype(np.float64))
    assert np.allclose(sums[0].cpu().numpy(), want, rtol=2e-5)
    h_out = h_in + I.normal(h_in.shape, 0.3, (47,))
    resid = torch.zeros((1, m.n_v, m.hidden), dtype=mdt, device=dev)
    say("edge cache_store", name)
    api.dc_cache_store(cfg, t(h_out[None], dev), t(h_in[None], dev), resid, [0])
    torch.cuda.synchronize()
    exact = (h_out[: m.n_v].astype(np.float64) - h_in[: m.n_v]).astype(np.float32)
    assert np.array_equal(resid[0].float().cpu().numpy(), I.round_bf16(exact) if _bf(m) else exact)


def test_empty_index_lists_leave_buffers_untouched(api, dev):
    """Every per-sample entry point with an empty index list is a no-op."""
    import torch
    m, cid = EDGE["bf16-N111"]
    W = I.Weights(m, cid)
    cfg = api.model_cfg(m)
    dmb = api.DeviceModel(_OneBlock(W, 0), dev)
    dmh = api.DeviceModel(_Head(W), dev)
    ws = api.Workspace(m, 1, dev)
    h = torch.full((1, m.n_tok, m.hidden), 3.0, device=dev)
    x = torch.full((1, m.lat_c, m.lat_t, m.lat_h, m.lat_w), 5.0, device=dev)
    txt = torch.zeros((1, m.n_txt, m.hidden), device=dev)
    r = torch.full((1, m.n_v, m.hidden), 2.0, device=dev, dtype=torch.bfloat16)
    g = torch.full((1, m.n_v, m.hidden), 4.0, device=dev)
    sums = torch.full((1, 4), 6.0, dtype=torch.float64, device=dev)
    mod = torch.zeros((6, m.hidden), device=dev)
    say("empty index lists")
    api.dc_patch_embed(dmh, x, txt, h, [], ws)
    api.dc_block_forward(dmb, 0, mod, h, [], ws)
    api.dc_cache_store(cfg, h, h, r, [])
    api.dc_cache_apply(cfg, h, r, g, [])
    api.dc_drift_l1(cfg, h, mod[:2], r, 0, sums, [], ws)
    api.dc_drift_l1(cfg, h, mod[:2], r, 1, sums, [], ws)
    api.dc_head_euler(dmh, mod[:2], g, x, 0.5, [], ws)
    torch.cuda.synchronize()
    assert (h == 3.0).all() and (x == 5.0).all() and (r.float() == 2.0).all()
    assert (g == 4.0).all() and (sums == 6.0).all()


class _AttentionOnly:
    """Block 0 of W reduced to its attention: query rows of W_qkv multiplied by a power of
    two (exact in bf16), W_o = I and b_o = 0, so with gate1 = 1 and gate2 = 0 the block
    adds the attention output itself to h."""

    def __init__(self, W, factor):
        self.W, self.f = W, factor
        self.m = W.m

    def get(self, name):
        return self.W.get(name)

    def block(self, l, name):
        d = self.m.hidden
        if name == "w_o":
            return np.eye(d, dtype=np.float32)
        if name == "b_o":
            return np.zeros(d, np.float32)
        a = self.W.block(l, name)
        if name == "w_qkv":
            a = a.copy()
            a[:d] *= self.f
        return a


def test_attention_large_logits(api, dev):
    """8,269 tokens x 30 heads of 64 run the long-sequence attention kernel.  Query
    weights scaled by 64 spread the logits of a row over hundreds of log2 units: a
    later key tile lies far above the first tile's maximum, so the fast pass raises
    its running maximum or, past the fp32 range, the workgroup redoes the item with
    the tile maximum on every tile.  The block is reduced to its attention (W_o = I,
    gate1 = 1, gate2 = 0).  The logits are so steep that rounding q and k to bf16
    decides which key dominates, so the reference takes a, q, k and v rounded to
    bf16 at the points where the device rounds them (q after its log2(e)/sqrt(d_h)
    scale), then the oracle's attention; sampled rows."""
    import math
    import torch
    m = _shape(1920, 30, 64, 7680, (16, 32, 64), 77, "bf16")
    assert m.n_tok >= 8192
    d = m.hidden
    W = _AttentionOnly(I.Weights(m, 97), 64.0)
    dm = api.DeviceModel(W, dev)
    ws = api.Workspace(m, 1, dev)
    h = I.hidden_state(m, (42,))
    mod = mod_input(m, (43,))
    mod[2] = 1.0                          # gate1
    mod[5] = 0.0                          # gate2: no MLP
    dh = t(h[None], dev)
    say("large-logit attention N =", m.n_tok)
    api.dc_block_forward(dm, 0, t(mod, dev), dh, [0], ws)
    torch.cuda.synchronize()
    got = dh[0].cpu().numpy().astype(np.float64) - h
    assert np.isfinite(got).all()
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([[0, 1, 127, 128, m.n_v - 1, m.n_v, m.n_tok - 1],
                                     rng.integers(0, m.n_tok, 40)]))
    m64 = mod.astype(np.float64)
    a = I.round_bf16(dit.modulate(h.astype(np.float64), m64[0], m64[1], 1e-6).astype(np.float32))
    wqkv = W.block(0, "w_qkv").astype(np.float64)
    bqkv = W.block(0, "b_qkv").astype(np.float64)
    qkv = a.astype(np.float64) @ wqkv.T + bqkv
    qs = np.float32(1.4426950408889634 / math.sqrt(m.head_dim))
    q = I.round_bf16((qkv[rows, :d].astype(np.float32) * qs)).astype(np.float64)
    k = I.round_bf16(qkv[:, d: 2 * d].astype(np.float32)).astype(np.float64)
    v = I.round_bf16(qkv[:, 2 * d:].astype(np.float32)).astype(np.float64)
    # q k^T is in log2 units: scale q so the oracle's softmax(q k^T / sqrt(d_h)) is base 2
    want = dit.attention(q * (math.sqrt(m.head_dim) * math.log(2.0)), k, v, m.heads)
    err = rel_l2(got[rows], want)
    say("large-logit attention rel-L2", err)
    assert err < 1e-2


@pytest.mark.parametrize("name", ["bf16-N328", "bf16-N3597-h30-split"])
def test_head_rows_with_large_mean_and_outlier_first_value(api, dev, name):
    """The head's LayerNorm on rows whose mean is 40 standard deviations from zero, some
    with a first value 900 standard deviations from the mean: the LN statistics and the
    folded projection must not cancel catastrophically (the oracle is fp64)."""
    import torch
    m, cid = EDGE[name]
    W = I.Weights(m, cid)
    P = dit.Params(W)
    dm = api.DeviceModel(_Head(W), dev)
    ws = api.Workspace(m, 1, dev)
    x = I.latent(m, cid, 0)
    g = I.hidden_state(m, (44,))
    g[: m.n_v] += np.float32(40 * 0.16)
    g[: m.n_v: 7, 0] += np.float32(900 * 0.16)
    hm = mod_input(m, (45,))[:2]
    dx = t(x[None], dev)
    say("head large-mean rows", name)
    api.dc_head_euler(dm, t(hm, dev), t(g[None], dev), dx, -0.02, [0], ws)
    torch.cuda.synchronize()
    v = dit.head(P, hm.astype(np.float64), g[: m.n_v].astype(np.float64))
    want_x = dit.euler(x.astype(np.float64), v, 0.52, 0.5)
    got = dx[0].cpu().numpy()
    assert np.isfinite(got).all()
    err = rel_l2(got - x, want_x - x)
    say(name, "head update rel-L2 (large mean)", err)
    assert err < 1e-3
