"""The C-ABI library loads without a GPU and exports every function dc.h declares."""
import os
import re

import pytest

from paper_2608_16354_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "dc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\**\s+\**(dc_[a-z0-9_]+)\s*\(",
                                 src, flags=re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("dc_block_forward", "dc_cache_store", "dc_cache_apply", "dc_drift_l1",
              "dc_denoise_step", "dc_schedule_dp"):
        assert n in names
    assert set(names) == set(_lib.SIGNATURES), "binding and header disagree"


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_errors_are_reported_not_raised():
    import ctypes as C
    from paper_2608_16354_amd import api
    lib = _lib.load()
    assert lib.dc_schedule_dp(None, None) == _lib.DC_ERR_ARG
    assert b"NULL" in lib.dc_last_error()
    bad = _lib.ModelCfg(2, 250, 4, 64, 1024, 16, 4, 16, 16, 2, 16, 0, 1e-6)
    assert lib.dc_workspace_bytes(C.byref(bad), 1) == 0
    cfg = _lib.ModelCfg(2, 256, 4, 64, 1024, 16, 4, 16, 16, 2, 16, 0, 1e-6)
    assert lib.dc_workspace_bytes(C.byref(cfg), 1) > 0
    # a shape check fails before anything touches a device
    rc = lib.dc_block_forward(C.byref(bad), None, None, None, None, 0, None, 0, None)
    assert rc == _lib.DC_ERR_SHAPE


def test_sampler_options_are_validated_before_any_device_work():
    """dc_sampler_create_ex refuses bad legality options on the host (the pointers below
    are never dereferenced on the device: every case fails before the first device call)."""
    import ctypes as C
    import numpy as np
    from paper_2608_16354_amd import api
    from paper_2608_16354_amd import inputs as I
    lib = _lib.load()
    w = I.WORKLOADS["dit-tiny-f32"]
    m = w.model
    cfg = _lib.ModelCfg(m.n_blocks, m.hidden, m.heads, m.head_dim, m.mlp_hidden, m.lat_c, m.lat_t,
                        m.lat_h, m.lat_w, m.patch, m.n_txt, 0, m.ln_eps)
    fake = C.c_void_p(0x1000)
    blocks = (_lib.BlockWeights * m.n_blocks)()
    weights = _lib.ModelWeights()
    weights.blocks = C.cast(blocks, C.POINTER(_lib.BlockWeights))
    ws = lib.dc_workspace_bytes(C.byref(cfg), 2)
    bufs = _lib.Buffers(fake, fake, fake, fake, fake, fake, fake, fake, fake, ws)
    sig = np.ascontiguousarray(I.sigmas(w.K))
    sigp = sig.ctypes.data_as(C.POINTER(C.c_double))

    def create(problems, opts, B=1):
        cps = [api._CProblem(p) for p in problems]
        arr = (_lib.SchedProblem * len(cps))(*[c.c for c in cps])
        h = C.c_void_p()
        rc = lib.dc_sampler_create_ex(C.byref(cfg), C.byref(weights), B, arr, sigp, C.byref(bufs),
                                      C.byref(opts), None, C.byref(h))
        assert not h.value
        return rc, lib.dc_last_error()

    p = I.scene_problem(w, w.motions[0])
    # guidance: a non-finite scale, and more than half the batch limit
    o = _lib.SamplerOpts(); o.cfg = 1; o.guidance = float("nan"); o.txt_null = 0x1000
    assert create([p], o)[0] == _lib.DC_ERR_ARG
    o = _lib.SamplerOpts(); o.cfg = 1; o.guidance = 2.0; o.txt_null = 0x1000
    assert create([p] * 33, o, B=33)[0] == _lib.DC_ERR_ARG
    # two experts: k_switch out of range, no modulation table, no segment change
    low = _lib.ModelWeights()
    low.blocks = C.cast(blocks, C.POINTER(_lib.BlockWeights))
    o = _lib.SamplerOpts(); o.w_low = C.pointer(low); o.mod_low = 0x1000; o.k_switch = 1
    assert create([p], o)[0] == _lib.DC_ERR_ARG
    o.k_switch = w.K + 1
    assert create([p], o)[0] == _lib.DC_ERR_ARG
    o.k_switch = 5; o.mod_low = None
    assert create([p], o)[0] == _lib.DC_ERR_ARG
    o.mod_low = 0x1000
    rc, msg = create([p], o)
    assert rc == _lib.DC_ERR_ARG and b"segment" in msg
    # an unknown option value
    o = _lib.SamplerOpts(); o.cfg = 2
    assert create([p], o)[0] == _lib.DC_ERR_ARG


def test_calibration_and_noalloc_entry_points_validate_on_the_host():
    """dc_calibrate_tables and dc_drift_l1_noalloc refuse bad arguments before any device
    work (no GPU here: every case below must fail on the host)."""
    import ctypes as C
    lib = _lib.load()
    cfg = _lib.ModelCfg(2, 256, 4, 64, 1024, 16, 4, 16, 16, 2, 16, 0, 1e-6)
    assert lib.dc_calibrate_workspace_bytes(C.byref(cfg), 10) > 0
    assert lib.dc_calibrate_workspace_bytes(C.byref(cfg), 0) == 0
    q = (C.c_double * 18)()
    d = (C.c_double * 18)()
    sig = (C.c_double * 11)()
    rc = lib.dc_calibrate_tables(C.byref(cfg), None, None, None, sig, 10, 2, 1e-6, q, d, None, 0, None)
    assert rc == _lib.DC_ERR_ARG and b"NULL" in lib.dc_last_error()
    h72 = _lib.ModelCfg(2, 1152, 16, 72, 4608, 16, 4, 16, 16, 2, 16, 1, 1e-6)
    w = _lib.ModelWeights()
    fake = C.c_void_p(0x1000)
    rc = lib.dc_calibrate_tables(C.byref(h72), C.byref(w), fake, fake, sig, 10, 2, 1e-6, q, d, fake, 0, None)
    assert rc == _lib.DC_ERR_SHAPE
    idx = (C.c_int32 * 65)(*range(65))
    rc = lib.dc_drift_l1_noalloc(C.byref(cfg), fake, fake, fake, 0, fake, idx, 65, None)
    assert rc == _lib.DC_ERR_ARG
    rc = lib.dc_drift_l1_noalloc(C.byref(cfg), None, fake, fake, 0, fake, idx, 1, None)
    assert rc == _lib.DC_ERR_ARG
