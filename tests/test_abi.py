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
