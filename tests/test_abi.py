"""The C-ABI library loads on a host without a GPU, exports every declared symbol,
and rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2607_08642_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dominotree.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dt_[a-z_]+)\s*\(", text)))


def lib():
    assert os.path.exists(binding.LIB_PATH), "build first: python -c 'import __graft_entry__ as g; g.build()'"
    return binding.load()


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert set(names) == set(binding.EXPORTS)
    L = lib()
    for n in names:
        assert hasattr(L, n), n


def test_abi_version_and_status_strings():
    L = lib()
    assert L.dt_abi_version() == binding.ABI_VERSION
    for code in binding.STATUS:
        assert L.dt_status_string(code)
    assert L.dt_status_string(12345) == b"unknown status"


def test_null_arguments_rejected_on_host():
    L = lib()
    assert L.dt_plan_create(None, None, 1, 1, None, None, 0, 1, 1, 1, 0, 1, None) == -1
    h = ctypes.c_void_p(1)
    assert L.dt_plan_create(ctypes.byref(h), None, 1, 1, None, None, 0, 1, 1, 1, 0, 1, None) == -1
    assert h.value is None        # *plan is cleared on failure
    assert b"required" in L.dt_last_error()
    assert L.dt_workspace_size(None, 1, None) == -1
    assert L.dt_build_tree(None, None, 1, None, 0.0, None, 0, None, None) == -1
    L.dt_plan_destroy(None)
    # the model and the plan made from one
    m = ctypes.c_void_p(1)
    assert L.dt_model_create(None, None, 1, 1, None, None, 0) == -1
    assert L.dt_model_create(ctypes.byref(m), None, 1, 1, None, None, 0) == -1
    assert m.value is None
    h = ctypes.c_void_p(1)
    assert L.dt_plan_create_from_model(ctypes.byref(h), None, 4, 8, 8, 0, 1, None) == -1
    assert h.value is None and b"model" in L.dt_last_error()
    assert L.dt_plan_create_from_model(None, None, 4, 8, 8, 0, 1, None) == -1
    L.dt_model_destroy(None)


def test_bad_shapes_and_dtypes_rejected_on_host():
    L = lib()
    gru = binding.dt_gru(8, 8, None, None, 64, 64)
    head = binding.dt_head(8, None)
    h = ctypes.c_void_p()
    # dtype code
    assert L.dt_plan_create(ctypes.byref(h), 16, 100, 64, ctypes.byref(gru), ctypes.byref(head),
                            7, 4, 8, 8, 0, 1, None) == -3
    # M > V
    assert L.dt_plan_create(ctypes.byref(h), 16, 10, 64, ctypes.byref(gru), ctypes.byref(head),
                            0, 4, 11, 8, 0, 1, None) == -2
    # d_in != d_e
    gru2 = binding.dt_gru(8, 8, None, None, 32, 64)
    assert L.dt_plan_create(ctypes.byref(h), 16, 100, 64, ctypes.byref(gru2), ctypes.byref(head),
                            0, 4, 8, 8, 0, 1, None) == -2
    # envelope: d_h not a multiple of 32, B too large
    gru3 = binding.dt_gru(8, 8, None, None, 64, 48)
    assert L.dt_plan_create(ctypes.byref(h), 16, 100, 64, ctypes.byref(gru3), ctypes.byref(head),
                            0, 4, 8, 8, 0, 1, None) == -4
    assert L.dt_plan_create(ctypes.byref(h), 16, 1000, 64, ctypes.byref(gru), ctypes.byref(head),
                            0, 4, 8, 257, 0, 1, None) == -4
    # options
    bad = binding.dt_options(0, 5, 0, 0)
    assert L.dt_plan_create(ctypes.byref(h), 16, 100, 64, ctypes.byref(gru), ctypes.byref(head),
                            0, 4, 8, 8, 0, 1, ctypes.byref(bad)) == -4
    # alignment of the embedding table
    assert L.dt_plan_create(ctypes.byref(h), 18, 100, 64, ctypes.byref(gru), ctypes.byref(head),
                            0, 4, 8, 8, 0, 1, None) == -6
    assert h.value is None
    # the same checks on the model alone
    m = ctypes.c_void_p()
    assert L.dt_model_create(ctypes.byref(m), 16, 100, 64, ctypes.byref(gru), ctypes.byref(head), 7) == -3
    assert L.dt_model_create(ctypes.byref(m), 16, 100, 64, ctypes.byref(gru2), ctypes.byref(head), 0) == -2
    assert L.dt_model_create(ctypes.byref(m), 16, 100, 64, ctypes.byref(gru3), ctypes.byref(head), 0) == -4
    assert L.dt_model_create(ctypes.byref(m), 18, 100, 64, ctypes.byref(gru), ctypes.byref(head), 0) == -6
    assert m.value is None


def test_scan_workspace_query_and_checks():
    L = lib()
    n = ctypes.c_size_t()
    assert L.dt_scan_workspace_size(16, 151936, 64, ctypes.byref(n)) == 0 and n.value > 0
    assert L.dt_scan_workspace_size(16, 10, 64, ctypes.byref(n)) == -2
    assert L.dt_scan_workspace_size(16, 1000, 300, ctypes.byref(n)) == -4
    assert L.dt_scan_topm(16, 4, 100, 0, 8, 0.0, 16, 16, 16, 16, None, 0, None) == -5
    assert L.dt_scan_topm(16, 4, 100, 0, 8, 0.0, 16, 16, 16, 16, 256 + 16, 1 << 30, None) == -6
