"""The C-ABI library on a host without a GPU: it loads, exports every entry
point that include/rrf.h declares, and rejects bad arguments before touching
the device.  No compute call is made here."""

import ctypes
import os
import re

import pytest

from paper_2608_28941_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rrf.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rrf_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = _abi.load()
    names = declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(lib, name), name
    # The binding declares exactly the header's functions.
    assert sorted(_abi.SIGNATURES) == names


def test_status_strings():
    lib = _abi.load()
    for code in (0, 1, -1, -2, -3, -4, -5, -6, 42):
        s = lib.rrf_status_string(code)
        assert s and s.startswith(b"RRF")


def test_workspace_size_host_only():
    lib = _abi.load()
    out = ctypes.c_size_t()
    assert lib.rrf_workspace_size(1, 16384, 16384, 64, 0, ctypes.byref(out)) == 0
    # Bws alone is 16384^2 doubles.
    assert out.value >= 16384 * 16384 * 8 * 3
    # Blocks of up to 128 columns (run as 64-column sub-blocks).
    assert lib.rrf_workspace_size(1, 100, 50, 128, 0, ctypes.byref(out)) == 0
    assert lib.rrf_workspace_size(1, 16384, 16384, 64, 0, ctypes.byref(out)) == 0
    small = ctypes.c_size_t()
    assert lib.rrf_workspace_size(0, 100, 50, 16, 10, ctypes.byref(small)) == 0
    assert 0 < small.value < out.value
    for bad in [(2, 10, 10, 8, 0), (1, 0, 10, 8, 0), (1, 10, 10, 0, 0),
                (1, 10, 10, 129, 0), (1, 10, 10, 8, -1)]:
        assert lib.rrf_workspace_size(*bad, ctypes.byref(out)) == _abi.RRF_ERR_INVALID_ARG
    assert lib.rrf_workspace_size(1, 10, 10, 8, 0, None) == _abi.RRF_ERR_INVALID_ARG


def test_invalid_arguments_rejected_before_device():
    lib = _abi.load()
    h = ctypes.c_void_p()
    E = _abi.RRF_ERR_INVALID_ARG
    assert lib.rrf_plan_create(None, 1, 10, 10, 8, 0, None) == E
    assert lib.rrf_plan_create(ctypes.byref(h), 7, 10, 10, 8, 0, None) == E
    assert lib.rrf_plan_create(ctypes.byref(h), 1, 0, 10, 8, 0, None) == E
    assert lib.rrf_plan_create(ctypes.byref(h), 1, 10, 10, 129, 0, None) == E
    q, b = ctypes.c_void_p(), ctypes.c_void_p()
    l1, l2, k = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(7)
    assert lib.rrf_run(None, ctypes.c_void_p(8), 4, 4, 4, 0.1, 2, 1,
                       ctypes.byref(q), ctypes.byref(l1), ctypes.byref(k),
                       ctypes.byref(b), ctypes.byref(l2)) == E
    assert k.value == 7   # outputs untouched on error
    assert lib.rrf_destroy(None) == _abi.RRF_OK
    assert lib.rrf_set_timing(None, 1) == E
    assert lib.rrf_set_stop_mode(None, 0) == E
    nb = ctypes.c_int64()
    assert lib.rrf_get_trace(None, 0, ctypes.byref(nb), None, None, None, None, None) == E
    assert lib.rrf_set_power_iterations(None, 1) == E
    assert lib.rrf_sketch(1, 0, -1, 0, 1, ctypes.c_void_p(8), 1, None) == E
    assert lib.rrf_sketch(1, 0, 10, 0, 1, None, 10, None) == E
    assert lib.rrf_sketch(1, 0, 10, 0, 1, ctypes.c_void_p(8), 5, None) == E
    assert lib.rrf_sketch(1, 0, 0, 0, 0, ctypes.c_void_p(8), 1, None) == _abi.RRF_OK
    assert lib.rrf_copy_matrix(1, None, 1, ctypes.c_void_p(8), 1, 1, 1, None) == E
    assert lib.rrf_panel_qr(None, None, 4, 2, 4, None, 4, None, 2, None) == E
    assert lib.rrf_apply_block_reflector(None, 1, None, 4, None, 2, 2, None, 4,
                                         4, 4) == E
    assert lib.rrf_subspace_map(None, ctypes.c_void_p(8), 4, 2, ctypes.c_void_p(8), 4, 2,
                                ctypes.c_void_p(8), 2, 4, 3, ctypes.c_void_p(8), 2) == E
    p8 = ctypes.c_void_p(8)
    assert lib.rrf_panel_qr_noalloc(1, None, 100, 8, 100, p8, 100, p8, 8, p8, None,
                                    None) == E
    assert lib.rrf_panel_qr_noalloc(3, p8, 100, 8, 100, p8, 100, p8, 8, p8, None, None) == E
    assert lib.rrf_panel_qr_noalloc(1, p8, 100, 8, 100, p8, 100, p8, 7, p8, None, None) == E
    assert lib.rrf_panel_qr_noalloc(1, p8, 7, 8, 100, p8, 100, p8, 8, p8, None, None) == E
    # Beyond the static scratch: rejected before any device call.
    assert lib.rrf_panel_qr_noalloc(1, p8, 20000, 8, 20000, p8, 20000, p8, 8, p8, None,
                                    None) == _abi.RRF_ERR_SHAPE


def test_plan_create_without_gpu_reports_hip_error():
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:
        has_gpu = False
    if has_gpu:
        pytest.skip("a GPU is present")
    lib = _abi.load()
    h = ctypes.c_void_p()
    assert lib.rrf_plan_create(ctypes.byref(h), 1, 10, 10, 8, 0, None) == _abi.RRF_ERR_HIP
    assert not h.value


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_abi, "_lib", None)
    monkeypatch.setattr(_abi, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        _abi.load()


def test_caller_workspace_checked_before_device():
    # rrf_plan_create_in: a misaligned or short workspace is rejected on the
    # host, before any device call (the pointer is never dereferenced).
    lib = _abi.load()
    h = ctypes.c_void_p()
    need = ctypes.c_size_t()
    assert lib.rrf_workspace_size(1, 300, 200, 16, 0, ctypes.byref(need)) == 0
    args = (ctypes.byref(h), 1, 300, 200, 16, 0, None)
    assert lib.rrf_plan_create_in(*args, ctypes.c_void_p(0x1000 + 8),
                                  need.value) == _abi.RRF_ERR_INVALID_ARG
    assert lib.rrf_plan_create_in(*args, ctypes.c_void_p(0x100000),
                                  need.value - 1) == _abi.RRF_ERR_INVALID_ARG
    assert lib.rrf_plan_create_in(None, 1, 300, 200, 16, 0, None,
                                  ctypes.c_void_p(0x100000), need.value) == _abi.RRF_ERR_INVALID_ARG
    assert h.value is None
