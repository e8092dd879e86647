"""rrf_panel_qr_noalloc (the entry point for callers that cannot allocate)
against rrf_panel_qr, through the C ABI.

Two calls in a row on the same GPU (the second with a smaller panel, so the
static scratch still holds the first call's contents), both dtypes.  The bar
is the panel stage's: Householder QR is backward stable, so with cond(Y) =
100 the reflectors of the two entry points agree to ~cond * u; the wait flag
must read 0.
"""

import ctypes

import numpy as np
import pytest

import workloads as W
from tests.gpu_util import say, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2608_28941_amd as rrf  # noqa: E402
from paper_2608_28941_amd import _abi  # noqa: E402


def _noalloc(Y, dtype_code, stream):
    lib = _abi.load()
    m, b = Y.shape
    tdt = Y.dtype
    V = torch.full((b, m), float("nan"), dtype=tdt, device="cuda").t()
    T = torch.full((b, b), float("nan"), dtype=tdt, device="cuda").t()
    tau = torch.full((b,), float("nan"), dtype=tdt, device="cuda")
    flag = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    st = lib.rrf_panel_qr_noalloc(
        dtype_code, ctypes.c_void_p(Y.data_ptr()), m, b, Y.stride(1),
        ctypes.c_void_p(V.data_ptr()), m, ctypes.c_void_p(T.data_ptr()), b,
        ctypes.c_void_p(tau.data_ptr()), ctypes.c_void_p(flag.data_ptr()),
        ctypes.c_void_p(stream.cuda_stream))
    assert st == _abi.RRF_OK, _abi.status_string(st)
    return V, T, tau, flag


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_noalloc_panel_matches_panel_qr(dtype):
    tdt = torch.float64 if dtype == np.float64 else torch.float32
    code = _abi.RRF_F64 if dtype == np.float64 else _abi.RRF_F32
    stream = torch.cuda.current_stream()
    tol = 100 * 100 * np.finfo(dtype).eps
    for (m, b, seed) in [(16384, 64, 21), (3001, 37, 22)]:
        say(f"noalloc panel dtype={np.dtype(dtype).name} m={m} b={b}")
        Yh = W.random_graded(m, b, dtype, seed, decay=1e-2)
        Y = to_dev(Yh)
        V, T, tau, flag = _noalloc(Y, code, stream)
        with rrf.Plan(tdt, m, b, b) as p:
            V0, T0, tau0 = p.panel_qr(Y)
        V, T, tau = to_host(V), to_host(T), to_host(tau)
        V0, T0, tau0 = to_host(V0), to_host(T0), to_host(tau0)
        assert int(flag.item()) == 0
        assert np.all(np.isfinite(V)) and np.all(np.isfinite(T)) and np.all(np.isfinite(tau))
        assert np.max(np.abs(tau - tau0)) < tol
        assert np.max(np.abs(V - V0)) < tol * max(1.0, np.max(np.abs(V0)))
        assert np.max(np.abs(T - T0)) < tol * np.max(np.abs(T0))
        assert np.all(np.tril(T, -1) == 0)
        assert np.all(np.triu(V, 1) == 0) and np.all(np.diag(V) == 1)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    lib = _abi.load()
    p = ctypes.c_void_p(8)
    s = ctypes.c_void_p(0)
    assert lib.rrf_panel_qr_noalloc(1, p, 16385, 64, 16385, p, 16385, p, 64, p, None, s) \
        == _abi.RRF_ERR_SHAPE
    assert lib.rrf_panel_qr_noalloc(1, p, 1000, 65, 1000, p, 1000, p, 65, p, None, s) \
        == _abi.RRF_ERR_INVALID_ARG
    assert lib.rrf_panel_qr_noalloc(1, p, 1000, 64, 999, p, 1000, p, 64, p, None, s) \
        == _abi.RRF_ERR_INVALID_ARG
