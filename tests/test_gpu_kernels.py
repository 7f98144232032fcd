"""Device steps of the hot path against the oracle, through the C ABI.

Sizes: the small fp32 model, the 12-block bf16 model (several tiles and a
ragged tail: N = 3,704 tokens, head_dim 72), and the full 30- and 42-block
shapes (17,776 tokens) in the launch configuration the benchmark uses, where
the oracle computes sampled rows."""
import numpy as np
import pytest

from oracle import dit, runtime
from paper_2608_16354_amd import inputs as I
from tests.gpu_util import mod_input, rel_l2, say, t

pytestmark = pytest.mark.gpu

SMALL = ["dit-tiny-f32", "dit-12x1152-bf16"]
ALL = SMALL + ["dit-30x1920-bf16", "dit-42x3072-bf16"]


@pytest.fixture(scope="module")
def api():
    from paper_2608_16354_amd import api as A
    A.L.load()
    return A


def _bf(m):
    return m.dtype == "bf16"


@pytest.mark.parametrize("name", SMALL + ["dit-30x1920-bf16"])
def test_cache_store_and_apply_bit_exact(api, dev, name):
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    cfg = api.model_cfg(m)
    B = 3
    h_in = I.normal((B, m.n_tok, m.hidden), 1.0, (8000, 1))
    h_out = h_in + I.normal((B, m.n_tok, m.hidden), 0.3, (8000, 2))
    mdt = torch.bfloat16 if _bf(m) else torch.float32
    resid = torch.zeros((B, m.n_v, m.hidden), dtype=mdt, device=dev)
    say("cache_store", name)
    api.dc_cache_store(cfg, t(h_out, dev), t(h_in, dev), resid, [0, 2])
    torch.cuda.synchronize()
    # r = h_out - h_in (one fp32 subtraction, then round-to-nearest-even to bf16)
    exact = (h_out[:, : m.n_v].astype(np.float64) - h_in[:, : m.n_v]).astype(np.float32)
    want = I.round_bf16(exact) if _bf(m) else exact
    got = resid.float().cpu().numpy()
    assert np.array_equal(got[[0, 2]], want[[0, 2]])
    assert not got[1].any()                        # unselected sample untouched
    say("cache_apply", name)
    g = torch.full((B, m.n_tok, m.hidden), 7.0, device=dev)
    api.dc_cache_apply(cfg, t(h_in, dev), resid, g, [2])
    torch.cuda.synchronize()
    gg = g.cpu().numpy()
    want_g = (h_in[2, : m.n_v].astype(np.float64) + want[2]).astype(np.float32)
    assert np.array_equal(gg[2, : m.n_v], want_g)
    assert (gg[2, m.n_v:] == 7.0).all() and (gg[[0, 1]] == 7.0).all()


@pytest.mark.parametrize("name", ALL)
def test_drift_sums_and_snapshot(api, dev, name):
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    cfg = api.model_cfg(m)
    ws = api.Workspace(m, 2, dev)
    B = 2
    h_in = np.stack([I.hidden_state(m, (10, b)) for b in range(B)])
    mod0 = mod_input(m, (11,))[:2]
    mdt = torch.bfloat16 if _bf(m) else torch.float32
    u_ref = torch.zeros((B, m.n_v, m.hidden), dtype=mdt, device=dev)
    sums = torch.zeros((B, 4), dtype=torch.float64, device=dev)
    dh = t(h_in, dev)
    dmod = t(mod0, dev)
    say("drift snapshot", name)
    api.dc_drift_l1(cfg, dh, dmod, u_ref, 1, None, [0, 1], ws)
    torch.cuda.synchronize()
    u = [dit.modulate(h_in[b, : m.n_v].astype(np.float64), mod0[0].astype(np.float64),
                      mod0[1].astype(np.float64), m.ln_eps) for b in range(B)]
    got = u_ref.float().cpu().numpy().astype(np.float64)
    for b in range(B):
        if _bf(m):
            # the device rounds its fp32 u to bf16: within one bf16 ulp of the rounded oracle value
            ulp = np.abs(I.round_bf16(u[b].astype(np.float32))).astype(np.float64) * 2.0 ** -7
            assert (np.abs(got[b] - u[b]) <= ulp + 1e-6).all()
        else:
            assert np.abs(got[b] - u[b]).max() < 1e-5
    # compare mode against a seeded reference (the generator's, not the device's)
    ref = I.normal((B, m.n_v, m.hidden), 1.0, (12,))
    ref = I.round_bf16(ref) if _bf(m) else ref
    u_ref.copy_(t(ref, dev, mdt))
    say("drift compare", name)
    api.dc_drift_l1(cfg, dh, dmod, u_ref, 0, sums, [0, 1], ws)
    torch.cuda.synchronize()
    s1 = sums.cpu().numpy().copy()
    api.dc_drift_l1(cfg, dh, dmod, u_ref, 0, sums, [0, 1], ws)
    torch.cuda.synchronize()
    assert np.array_equal(s1, sums.cpu().numpy())        # bitwise reproducible
    for b in range(B):
        want = runtime.drift_sums(u[b], ref[b].astype(np.float64))
        assert np.allclose(s1[b], want, rtol=2e-5), (s1[b], want)
        assert runtime.drift_value(s1[b], 1e-6) == pytest.approx(runtime.drift_value(want, 1e-6), rel=2e-5)


@pytest.mark.parametrize("name", SMALL + ["dit-30x1920-bf16"])
def test_patch_embed(api, dev, name):
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    W = I.Weights(m, w.cfg_id)
    say("upload", name)
    dm = api.DeviceModel(W, dev)
    ws = api.Workspace(m, 2, dev)
    x = np.stack([I.latent(m, w.cfg_id, s) for s in range(2)])
    txt = np.stack([I.text(m, w.cfg_id, s) for s in range(2)])
    h_in = torch.zeros((2, m.n_tok, m.hidden), device=dev)
    say("patch_embed", name)
    api.dc_patch_embed(dm, t(x, dev), t(txt, dev), h_in, [1], ws)
    torch.cuda.synchronize()
    got = h_in.cpu().numpy()
    P = dit.Params(W)
    want = dit.embed(P, x[1], txt[1])
    # fp32 model: fp32 SIMT GEMM.  bf16 model: the fp32 operands are split into two
    # bf16 terms each (16 significand bits), so about 2^-18 relative per product;
    # the bf16 model's own bar is 1e-2 per block.
    tol = 1e-5 if m.dtype == "bf16" else 1e-6
    assert rel_l2(got[1, : m.n_v], want[: m.n_v]) < tol
    assert np.array_equal(got[1, m.n_v:], txt[1])
    assert not got[0].any()


@pytest.mark.parametrize("name", SMALL)
def test_time_modulation(api, dev, name):
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    W = I.Weights(m, w.cfg_id)
    dm = api.DeviceModel(W, dev)
    ws = api.Workspace(m, 1, dev)
    sig = I.sigmas(w.K)
    mod = torch.zeros((w.K, m.n_blocks + 1, 6, m.hidden), device=dev)
    say("time_modulation", name)
    api.dc_time_modulation(dm, sig[: w.K], mod, ws)
    torch.cuda.synchronize()
    got = mod.cpu().numpy()
    P = dit.Params(W)
    for k in range(w.K):
        blocks, head = dit.step_modulation(P, sig[k])
        for l in range(m.n_blocks):
            assert rel_l2(got[k, l], blocks[l]) < 1e-5
        assert rel_l2(got[k, m.n_blocks, :2], head) < 1e-5
        assert not got[k, m.n_blocks, 2:].any()


@pytest.mark.parametrize("name", ALL)
def test_block_forward(api, dev, name):
    """One block in place on a seeded residual stream.  Full comparison for the
    small models; for the 17,776-token models the oracle computes sampled rows
    (spanning video and text, first and last tiles)."""
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    W = I.Weights(m, w.cfg_id)
    l = m.n_blocks - 1
    for nm in ("w_qkv", "w_o", "w_1", "w_2"):
        W.block(l, nm)
    say("upload", name)
    dm = api.DeviceModel(_OneBlock(W, l), dev)
    ws = api.Workspace(m, 1, dev)
    h = I.hidden_state(m, (20,))
    mod = mod_input(m, (21,))
    dh = t(h[None], dev)
    say("block_forward", name, "N =", m.n_tok)
    api.dc_block_forward(dm, 0, t(mod, dev), dh, [0], ws)
    torch.cuda.synchronize()
    got = dh[0].cpu().numpy()
    P = dit.Params(W)
    big = m.n_tok > 5000
    rows = None
    if big:
        rng = np.random.default_rng(0)
        rows = np.unique(np.concatenate([[0, 1, 127, 128, m.n_v - 1, m.n_v, m.n_tok - 1],
                                         rng.integers(0, m.n_tok, 40)]))
    want = dit.block(P, l, mod.astype(np.float64), h.astype(np.float64), rows=rows)
    ref_in = h if rows is None else h[rows]
    gsel = got if rows is None else got[rows]
    err_h = rel_l2(gsel, want)
    err_d = rel_l2(gsel - ref_in, want - ref_in)
    say(name, "block rel-L2 h_out", err_h, "update", err_d)
    if _bf(m):
        assert err_h < 1e-2 and err_d < 2e-2
    else:
        assert err_h < 1e-5 and err_d < 1e-5


class _OneBlock:
    """A `Weights` view exposing block l as the model's only block."""

    def __init__(self, W, l):
        self.W, self.l = W, l
        self.m = W.m.__class__(**{**W.m.__dict__, "n_blocks": 1})

    def get(self, name):
        return self.W.get(name)

    def block(self, l, name):
        return self.W.block(self.l, name)


def _head_tol(m):
    """The bf16 head with d <= 2048 is the fused one-pass kernel, which feeds the matrix
    cores split (hi + lo) bf16 operands and so stays near fp32 accuracy; wider bf16 models
    take LN-modulation to bf16 rows, then the GEMM."""
    if not _bf(m):
        return 1e-5
    return 1e-4 if m.hidden <= 2048 else 1e-2


@pytest.mark.parametrize("name", ALL)
def test_head_euler(api, dev, name):
    import torch
    w = I.WORKLOADS[name]
    m = w.model
    W = I.Weights(m, w.cfg_id)
    dm = api.DeviceModel(_Head(W), dev)
    ws = api.Workspace(m, 1, dev)
    g = I.hidden_state(m, (30,))
    x = I.latent(m, w.cfg_id, 0)
    hm = mod_input(m, (31,))[:2]
    dx = t(x[None], dev)
    say("head_euler", name)
    api.dc_head_euler(dm, t(hm, dev), t(g[None], dev), dx, -0.02, [0], ws)
    torch.cuda.synchronize()
    got = dx[0].cpu().numpy()
    P = dit.Params(W)
    v = dit.head(P, hm.astype(np.float64), g[: m.n_v].astype(np.float64))
    want = dit.euler(x.astype(np.float64), v, 0.52, 0.5)
    err = rel_l2(got - x, want - x)
    say(name, "head update rel-L2", err)
    assert err < _head_tol(m)


class _Head:
    """Global weights only (the head test needs no blocks)."""

    def __init__(self, W):
        self.W = W
        self.m = W.m.__class__(**{**W.m.__dict__, "n_blocks": 1})

    def get(self, name):
        return self.W.get(name)

    def block(self, l, name):
        shapes = I.tensor_shapes(self.m)[1]
        return np.zeros(shapes[name], np.float32)
