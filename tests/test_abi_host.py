"""Host-only checks of the C-ABI library: it loads without a GPU and exports
every function include/gwtf_mcf.h declares (no compute call is made)."""
import ctypes
import os
import re

import pytest

from paper_2509_21221_amd import mcf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gwtf_mcf.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gwtf_(?:mcf|whatif)_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("gwtf_mcf_create", "gwtf_mcf_solve_batch", "gwtf_mcf_get_flows",
                     "gwtf_mcf_destroy", "gwtf_whatif_count", "gwtf_mcf_whatif_expand",
                     "gwtf_mcf_whatif_best"):
        assert required in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(mcf.LIB_PATH):
        pytest.fail("libgwtf_mcf.so not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(mcf.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_names_match_header():
    for name in declared_functions():
        assert callable(getattr(mcf, name)), name


def test_header_constants_match_binding():
    text = open(HEADER).read()
    assert "GWTF_NO_ARC (-1)" in text and mcf.GWTF_NO_ARC == -1
    for name, value in [("GWTF_OK", 0), ("GWTF_ERR_INVALID_ARG", 1), ("GWTF_ERR_OUT_OF_MEMORY", 2),
                        ("GWTF_ERR_DEVICE", 3), ("GWTF_ERR_NOT_SOLVED", 4), ("GWTF_ERR_RANGE", 5),
                        ("GWTF_INST_OK", 0), ("GWTF_INST_BAD_INPUT", 1), ("GWTF_INST_OVERFLOW", 2),
                        ("GWTF_PASS_REGISTER", 1), ("GWTF_PASS_LDS", 2), ("GWTF_PASS_GRID", 3), ("GWTF_PASS_PACKED", 5),
                        ("GWTF_PASS_GLOBAL", 4)]:
        assert re.search(rf"\b{name}\s*=\s*{value}\b", text), name
        assert getattr(mcf, name) == value


def test_null_handle_calls_fail_cleanly():
    """Calls that reject their arguments before touching a device."""
    lib = mcf.load_library()
    assert lib.gwtf_mcf_solve_batch(None, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_get_flows(None, 0, 1, None, None, None, None, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_get_stats(None, 0, 1, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_get_passes(None, 0, 1, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_calibrate_handoff(0, None, 4, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_whatif_expand(None, None, None, 0, 1, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_whatif_best(None, 1, None, None, None, 0, 0, None) == mcf.GWTF_ERR_INVALID_ARG
    assert lib.gwtf_mcf_resolve_churn(None, None, None, None, None) == mcf.GWTF_ERR_INVALID_ARG
    assert "handle" in mcf.gwtf_mcf_last_error(None)
    lib.gwtf_mcf_destroy(None)
    out = ctypes.c_void_p(1)
    assert lib.gwtf_mcf_create(None, None, ctypes.byref(out)) == mcf.GWTF_ERR_INVALID_ARG
    assert out.value is None
    assert "shape" in mcf.gwtf_mcf_last_error(None)
    bad = mcf.gwtf_mcf_shape_t(0, 4, 1, 0)
    assert lib.gwtf_mcf_create(ctypes.byref(bad), None, ctypes.byref(out)) == mcf.GWTF_ERR_INVALID_ARG


def test_noalloc_solve_rejects_arguments_before_touching_a_device():
    lib = mcf.load_library()
    assert lib.gwtf_mcf_solve_batch_noalloc(None, None, None) == mcf.GWTF_ERR_INVALID_ARG
    assert "shape" in mcf.gwtf_mcf_last_error(None)
    shape = mcf.gwtf_mcf_shape_t(8, 8, 4, 0)
    assert lib.gwtf_mcf_solve_batch_noalloc(ctypes.byref(shape), None, None) == mcf.GWTF_ERR_INVALID_ARG
    assert "batch" in mcf.gwtf_mcf_last_error(None)
    b = mcf.gwtf_mcf_batch_t(5, 1, 1, 1, None, None, 1, 1, 1, 1)
    assert lib.gwtf_mcf_solve_batch_noalloc(ctypes.byref(shape), None, ctypes.byref(b)) == mcf.GWTF_ERR_INVALID_ARG
    assert "max_batch" in mcf.gwtf_mcf_last_error(None)
    b = mcf.gwtf_mcf_batch_t(2, 1, 1, None, None, None, 1, 1, 1, 1)
    assert lib.gwtf_mcf_solve_batch_noalloc(ctypes.byref(shape), None, ctypes.byref(b)) == mcf.GWTF_ERR_INVALID_ARG
    assert "arc_cost" in mcf.gwtf_mcf_last_error(None)


def test_product_path_fails_loudly_without_library(tmp_path):
    saved = mcf._lib
    mcf._lib = None
    try:
        with pytest.raises(RuntimeError, match="missing"):
            mcf.load_library(str(tmp_path / "nope.so"))
    finally:
        mcf._lib = saved


def test_whatif_count_is_host_only():
    """S!/(S-m)! placements, computed on the host (no device is touched)."""
    import math

    for S, m in [(1, 0), (1, 1), (4, 2), (8, 8), (12, 12), (20, 20), (64, 3)]:
        assert mcf.gwtf_whatif_count(S, m) == math.perm(S, m)
    for S, m in [(0, 0), (3, 4), (3, -1), (21, 21), (30, 20)]:
        with pytest.raises(mcf.GwtfError):
            mcf.gwtf_whatif_count(S, m)
    lib = mcf.load_library()
    assert lib.gwtf_whatif_count(4, 2, None) == mcf.GWTF_ERR_INVALID_ARG
