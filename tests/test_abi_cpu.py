"""The C-ABI library loads and exports every function include/fsx.h declares (CPU, no compute calls)."""

import ctypes
import os
import re

import pytest

from paper_2607_15621_amd import fsx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "fsx.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fsx_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("fsx_expert_create", "fsx_expert_forward", "fsx_cache_append_rows"):
        assert n in names
    assert set(names) == set(fsx.SYMBOLS)


def test_library_exports_every_declared_symbol():
    if not os.path.exists(fsx.LIB_PATH):
        pytest.fail("libfsx.so is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(fsx.LIB_PATH)
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_argument_checks_run_before_any_gpu_work():
    # These calls fail validation on the host and never reach the HIP runtime.
    L = fsx.lib()
    out = ctypes.c_void_p(1)
    assert L.fsx_expert_create(None, None, None, None, None, ctypes.byref(out)) == 1
    assert out.value is None
    assert "cfg" in fsx.last_error()
    bad = fsx.make_cfg(0, 512, 32, 128, 2048)
    assert L.fsx_expert_create(ctypes.byref(bad), None, None, None, None, ctypes.byref(out)) == 1
    bad = fsx.make_cfg(2, 512, 32, 128, 2048, max_batch=65)
    assert L.fsx_expert_create(ctypes.byref(bad), None, None, None, None, ctypes.byref(out)) == 1
    assert "max_batch" in fsx.last_error()
    assert L.fsx_expert_forward(None, None, None, 1, 0, None, None, None) == 1
    assert L.fsx_cache_append_rows(None, None, None, 4, 0, None) == 1
    assert fsx.version().count(".") == 2


def test_cache_layout_is_validated_before_any_gpu_work():
    import numpy as np

    lens = np.array([4], np.int64)
    desc = fsx.CacheDesc(None, None, fsx.BF16, 2, 4, 128, 8, lens)
    desc.c.layout = 7
    assert fsx.lib().fsx_cache_append_rows(ctypes.byref(desc.c), None, None, 4, 0, None) == 1
    assert "layout" in fsx.last_error()
    assert fsx.lib().fsx_probe_hbm_read(None, 16, 0, None, None) == 1
