"""The C-ABI library: loads, exports every declared entry point, and rejects
bad arguments on the host before touching a GPU (CPU-only tests)."""
from __future__ import annotations

import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lattice.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lattice_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_1912_05905_amd import lattice
    if not os.path.exists(lattice.LIB_PATH):
        pytest.fail("liblattice.so is not built (run __graft_entry__.build())")
    return lattice.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for need in ("lattice_create", "lattice_splat", "lattice_conv", "lattice_coarsen",
                 "lattice_refine", "lattice_slice", "lattice_deform_slice", "lattice_destroy",
                 "lattice_num_vertices", "lattice_export_keys", "lattice_export_neighbors",
                 "lattice_export_simplices", "lattice_distribute_pointnet", "lattice_splat_backward",
                 "lattice_slice_backward", "lattice_conv_backward", "lattice_deform_slice_backward", "lattice_conv_preact", "lattice_deform_slice_classify",
                 "lattice_refine_preact", "lattice_slice_and_deform", "lattice_coarsen_ex"):
        assert need in names


def test_every_declared_symbol_is_exported(lib):
    from paper_1912_05905_amd import lattice
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in lattice.SIGNATURES, f"binding lacks {name}"


def test_status_strings(lib):
    for code, name in {0: b"LAT_OK", -1: b"LAT_EINVAL", -4: b"LAT_EHASHFULL", -8: b"LAT_ELEVEL"}.items():
        assert lib.lattice_status_string(code) == name


def test_host_validation_without_gpu(lib):
    out = C.c_void_p()
    sigma = (C.c_float * 3)(0.1, 0.1, 0.1)
    assert lib.lattice_create(None, 10, 3, sigma, 0, None, None) == -1
    assert lib.lattice_create(None, 10, 2, sigma, 0, None, C.byref(out)) == -2
    assert b"d = 3" in lib.lattice_last_error()
    assert lib.lattice_create(None, -1, 3, sigma, 0, None, C.byref(out)) == -1
    assert lib.lattice_create(None, 10, 3, sigma, 0, None, C.byref(out)) == -1
    bad = (C.c_float * 3)(0.1, 0.0, 0.1)
    assert lib.lattice_create(C.c_void_p(16), 10, 3, bad, 0, None, C.byref(out)) == -1
    nan = (C.c_float * 3)(0.1, float("nan"), 0.1)
    assert lib.lattice_create(C.c_void_p(16), 10, 3, nan, 0, None, C.byref(out)) == -1
    assert lib.lattice_create(C.c_void_p(16), 10, 3, sigma, -5, None, C.byref(out)) == -1
    assert lib.lattice_create(C.c_void_p(16), 10, 3, None, 0, None, C.byref(out)) == -1
    assert out.value is None
    n = C.c_int64()
    assert lib.lattice_num_vertices(None, C.byref(n)) == -1
    assert lib.lattice_destroy(None) == 0
    assert lib.lattice_splat(None, None, 0, 8, 0, 1, None, 0, None, None) == -1
    assert lib.lattice_conv(None, None, None, 0, 8, None, None, 8, 0, 0, None, 0, None) == -1
    assert lib.lattice_refine(None, None, None, 0, 8, None, None, 8, 0, 0, None, 0, None) == -1
    assert lib.lattice_slice(None, None, 0, 8, 0, None, None) == -1
    assert lib.lattice_deform_slice(None, None, 0, 8, 0, None, 0.0, None, None, None) == -1
    assert lib.lattice_slice_and_deform(None, None, 0, 8, 0, None, 0.0, None, None, None) == -1
    assert lib.lattice_distribute_pointnet(None, None, None, 0, 4, None, None, C.c_float(1e-5), None, None, 16,
                                           None, None, 32, None, None, 64, 0, None, 0, None) == -1
    assert lib.lattice_coarsen(None, 0, None, C.byref(out)) == -1
    assert lib.lattice_coarsen_ex(None, 0, 0, None, C.byref(out)) == -1
    assert lib.lattice_splat_backward(None, None, 0, 8, 1, None, None, None) == -1
    assert lib.lattice_slice_backward(None, None, 0, 8, None, 0, None) == -1
    assert lib.lattice_conv_backward(None, None, None, 0, 8, None, 8, 0, None, 0, None, 0, None, 0, None, None,
                                     None) == -1
    assert lib.lattice_deform_slice_backward(None, None, 0, 8, None, 0.0, None, 0, None, 0, None, None, None) == -1


def test_timing_interface_without_events(lib):
    n = C.c_int64()
    ms = C.c_double()
    assert lib.lattice_timing_enable(b"conv", 1) == 0
    assert lib.lattice_timing_read(b"conv", C.byref(n), C.byref(ms)) == 0
    assert n.value == 0 and ms.value == 0.0
    assert lib.lattice_timing_enable(b"conv", 0) == 0
    assert lib.lattice_timing_read(b"never-used", C.byref(n), C.byref(ms)) == 0
