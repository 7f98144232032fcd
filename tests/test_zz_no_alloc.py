"""dc_drift_l1_noalloc (no workspace: the partial sums live in the library's fixed
per-GPU scratch array) against dc_drift_l1 with a caller workspace, through the C ABI.

Two calls in a row, the second on a smaller input (the 12-block shape with three
samples, then the small fp32 shape with one): the snapshot and the drift sums must
equal the workspace version's bit for bit (the same kernels in the same order).
"""
import numpy as np
import pytest

from paper_2608_16354_amd import inputs as I
from tests.gpu_util import say, t

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def api():
    from paper_2608_16354_amd import api as A
    A.L.load()
    return A


def _one_case(api, dev, name, B, idx, key):
    import torch
    m = I.WORKLOADS[name].model
    cfg = api.model_cfg(m)
    mdt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    h0 = t(I.normal((B, m.n_tok, m.hidden), 1.0, (8100, key, 0)), dev)
    h1 = t(I.normal((B, m.n_tok, m.hidden), 1.0, (8100, key, 1)), dev)
    h1[:, : m.n_v] = h1[:, : m.n_v] * 0.1 + h0[:, : m.n_v]              # a drift of about 10 %
    mod0 = t(I.normal((2, m.hidden), 0.1, (8100, key, 2)), dev)
    ws = api.Workspace(m, B, dev)
    u_ws = torch.zeros((B, m.n_v, m.hidden), dtype=mdt, device=dev)
    u_na = torch.full((B, m.n_v, m.hidden), 7.0, dtype=mdt, device=dev)
    s_ws = torch.full((B, 4), -1.0, dtype=torch.float64, device=dev)
    s_na = torch.full((B, 4), -2.0, dtype=torch.float64, device=dev)
    say("no-alloc drift snapshot", name, "B", B, "idx", idx)
    api.dc_drift_l1(cfg, h0, mod0, u_ws, 1, None, idx, ws)
    api.dc_drift_l1_noalloc(cfg, h0, mod0, u_na, 1, None, idx)
    torch.cuda.synchronize()
    for b in idx:
        assert torch.equal(u_ws[b], u_na[b])
    say("no-alloc drift compare", name)
    api.dc_drift_l1(cfg, h1, mod0, u_ws, 0, s_ws, idx, ws)
    api.dc_drift_l1_noalloc(cfg, h1, mod0, u_na, 0, s_na, idx)
    torch.cuda.synchronize()
    for b in idx:
        assert torch.equal(s_ws[b], s_na[b]), (b, s_ws[b], s_na[b])
        d = float(s_na[b, 0] / (s_na[b, 1] + 1e-6))
        assert 0.02 < d < 0.5
    unused = [b for b in range(B) if b not in idx]
    for b in unused:                                                    # untouched samples
        assert float(s_na[b, 0]) == -2.0
    return s_na.cpu().numpy()


def test_noalloc_drift_equals_workspace_drift_two_calls(api, dev):
    a = _one_case(api, dev, "dit-12x1152-bf16", 4, [3, 0, 2], 1)
    b = _one_case(api, dev, "dit-tiny-f32", 1, [0], 2)                 # smaller: fewer rows, one sample
    assert np.all(np.isfinite(a[[0, 2, 3]])) and np.all(np.isfinite(b))


def test_noalloc_drift_rejects_too_many_samples(api, dev):
    import torch
    m = I.WORKLOADS["dit-tiny-f32"].model
    cfg = api.model_cfg(m)
    h = torch.zeros((1, m.n_tok, m.hidden), device=dev)
    u = torch.zeros((1, m.n_v, m.hidden), device=dev)
    mod0 = torch.zeros((2, m.hidden), device=dev)
    sums = torch.zeros((1, 4), dtype=torch.float64, device=dev)
    with pytest.raises(api.L.DriveCacheError):
        api.dc_drift_l1_noalloc(cfg, h, mod0, u, 0, sums, list(range(api.L.DC_MAX_BATCH + 1)))
