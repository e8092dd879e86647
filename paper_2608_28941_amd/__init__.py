"""MI355X Householder blocked adaptive randomized range finder.

Python binding of librrf (include/rrf.h).  PyTorch provides device memory and
streams only; every step of the method runs in the library's HIP kernels.

    import torch, paper_2608_28941_amd as rrf
    A = torch.randn(4096, 4096, device="cuda", dtype=torch.float64)
    Q, B, k = rrf.run(A, tol=1e-2, block_b=32, seed=1)

Matrices cross the boundary column-major (LAPACK layout): a tensor of shape
(m, n) with strides (1, lda).  ``colmajor(t)`` makes such a copy.
"""

import ctypes

from . import _abi
from ._abi import (RRFError, RRF_F32, RRF_F64, RRF_OK, RRF_WARN_KMAX,
                   RRF_STOP_TRAILING, RRF_STOP_SUBTRACT, RRF_STOP_SPECTRAL, STAGES)

__all__ = ["Plan", "run", "sketch", "colmajor", "RRFError", "STAGES",
           "RRF_STOP_TRAILING", "RRF_STOP_SUBTRACT", "RRF_STOP_SPECTRAL"]


def _torch():
    import torch
    return torch


def _dtype_code(dt):
    torch = _torch()
    if dt == torch.float32:
        return RRF_F32
    if dt == torch.float64:
        return RRF_F64
    raise TypeError("only float32 and float64 are supported")


def _stream_handle(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def colmajor(t):
    """Column-major copy (strides (1, m)) of a 2-D CUDA tensor, or t itself."""
    if t.dim() != 2:
        raise ValueError("expected a matrix")
    if t.stride(0) == 1 and t.stride(1) >= max(1, t.shape[0]):
        return t
    return t.t().contiguous().t()


def _check_colmajor(t, name):
    if t.dim() != 2 or not t.is_cuda:
        raise ValueError(f"{name} must be a 2-D CUDA tensor")
    if t.numel() > 0 and t.shape[0] > 1 and t.stride(0) != 1:
        raise ValueError(f"{name} must be column-major (use colmajor())")
    return max(1, t.stride(1) if t.shape[1] > 1 else t.shape[0])


def _alloc_colmajor(m, n, ld, dtype, device):
    torch = _torch()
    buf = torch.empty(max(ld * n, 1), dtype=dtype, device=device)
    return buf.as_strided((m, n), (1, ld))


class Plan:
    """A plan (workspace for maxima m_max x n_max, block <= block_b_max)."""

    def __init__(self, dtype, m_max, n_max, block_b_max=64, k_max=0,
                 stream=None, device=None, workspace=None):
        """workspace: optional device tensor (any dtype, contiguous, 256-byte
        aligned, at least workspace_size(...) bytes) that the plan carves its
        device buffers from (rrf_plan_create_in); the plan keeps a reference
        to it."""
        torch = _torch()
        self.dtype = dtype
        self.code = _dtype_code(dtype)
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.stream = torch.cuda.current_stream(self.device) if stream is None else stream
        self.lib = _abi.load()
        h = ctypes.c_void_p()
        if workspace is None:
            st = self.lib.rrf_plan_create(ctypes.byref(h), self.code, int(m_max),
                                          int(n_max), int(block_b_max), int(k_max),
                                          _stream_handle(self.stream))
            _abi.check(st, "rrf_plan_create", allow_warn=False)
        else:
            if not workspace.is_cuda or not workspace.is_contiguous():
                raise ValueError("workspace must be a contiguous CUDA tensor")
            st = self.lib.rrf_plan_create_in(
                ctypes.byref(h), self.code, int(m_max), int(n_max), int(block_b_max),
                int(k_max), _stream_handle(self.stream),
                ctypes.c_void_p(workspace.data_ptr()),
                workspace.numel() * workspace.element_size())
            _abi.check(st, "rrf_plan_create_in", allow_warn=False)
        self.workspace = workspace
        self.handle = h
        self.m_max, self.n_max, self.block_b_max, self.k_max = (
            m_max, n_max, block_b_max, k_max)
        self.last_status = RRF_OK

    def close(self):
        if getattr(self, "handle", None):
            self.lib.rrf_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_stop_mode(self, mode):
        _abi.check(self.lib.rrf_set_stop_mode(self.handle, int(mode)),
                   "rrf_set_stop_mode")

    def set_power_iterations(self, q):
        _abi.check(self.lib.rrf_set_power_iterations(self.handle, int(q)),
                   "rrf_set_power_iterations")

    def set_timing(self, enable):
        _abi.check(self.lib.rrf_set_timing(self.handle, 1 if enable else 0),
                   "rrf_set_timing")

    def run_raw(self, A, tol, block_b, seed):
        """rrf_run on a column-major device tensor; returns the plan-owned
        device pointers (q_ptr, ldq, k, b_ptr, ldb) and the status."""
        if A.dtype != self.dtype:
            raise TypeError("A's dtype differs from the plan's")
        lda = _check_colmajor(A, "A")
        m, n = A.shape
        q = ctypes.c_void_p()
        b = ctypes.c_void_p()
        ldq = ctypes.c_int64()
        ldb = ctypes.c_int64()
        k = ctypes.c_int64()
        st = self.lib.rrf_run(self.handle, ctypes.c_void_p(A.data_ptr()), m, n,
                              lda, float(tol), int(block_b),
                              int(seed) & 0xFFFFFFFFFFFFFFFF,
                              ctypes.byref(q), ctypes.byref(ldq), ctypes.byref(k),
                              ctypes.byref(b), ctypes.byref(ldb))
        _abi.check(st, "rrf_run")
        self.last_status = st
        return q.value, ldq.value, k.value, b.value, ldb.value, st

    def _copy_out(self, ptr, ld, rows, cols, dtype=None):
        dtype = self.dtype if dtype is None else dtype
        out = _alloc_colmajor(rows, cols, max(rows, 1), dtype, self.device)
        if rows and cols:
            _abi.check(self.lib.rrf_copy_matrix(
                _dtype_code(dtype), ctypes.c_void_p(ptr), ld,
                ctypes.c_void_p(out.data_ptr()), max(rows, 1), rows, cols,
                _stream_handle(self.stream)), "rrf_copy_matrix")
        return out

    def run(self, A, tol, block_b, seed):
        """Alg. 2 + explicit Q.  Returns (Q, B, k) as new column-major tensors."""
        qp, ldq, k, bp, ldb, _ = self.run_raw(A, tol, block_b, seed)
        m, n = A.shape
        Q = self._copy_out(qp, ldq, m, k)
        B = self._copy_out(bp, ldb, k, n)
        return Q, B, k

    def trace(self):
        """Per-block (E_trail, E_sub, E_spec) of the last run, plus E0 and
        sigma^2."""
        nb = ctypes.c_int64()
        e0 = ctypes.c_double()
        s2 = ctypes.c_double()
        _abi.check(self.lib.rrf_get_trace(self.handle, 0, ctypes.byref(nb), None,
                                          None, None, ctypes.byref(e0),
                                          ctypes.byref(s2)),
                   "rrf_get_trace")
        cap = nb.value
        et = (ctypes.c_double * max(cap, 1))()
        es = (ctypes.c_double * max(cap, 1))()
        ep = (ctypes.c_double * max(cap, 1))()
        _abi.check(self.lib.rrf_get_trace(self.handle, cap, ctypes.byref(nb), et,
                                          es, ep, ctypes.byref(e0), ctypes.byref(s2)),
                   "rrf_get_trace")
        return {"E_trail": list(et)[:cap], "E_sub": list(es)[:cap],
                "E_spec": list(ep)[:cap], "E0": e0.value, "sigma2": s2.value,
                "nblocks": cap}

    def stage_stats(self):
        n = _abi.RRF_NUM_STAGES
        ms = (ctypes.c_double * n)()
        la = (ctypes.c_int64 * n)()
        fl = (ctypes.c_double * n)()
        by = (ctypes.c_double * n)()
        _abi.check(self.lib.rrf_get_stage_stats(self.handle, ms, la, fl, by),
                   "rrf_get_stage_stats")
        return {s: {"ms": ms[i], "launches": la[i], "flops": fl[i], "bytes": by[i]}
                for i, s in enumerate(STAGES)}

    def reflectors(self, m, k):
        """(V m x k, T (ldt rows) x k, tau k) of the last run, as float64
        copies (the library keeps reflectors in binary64 for both dtypes)."""
        torch = _torch()
        v = ctypes.c_void_p()
        t = ctypes.c_void_p()
        ta = ctypes.c_void_p()
        ldv = ctypes.c_int64()
        ldt = ctypes.c_int64()
        _abi.check(self.lib.rrf_get_reflectors(self.handle, ctypes.byref(v),
                                               ctypes.byref(ldv), ctypes.byref(t),
                                               ctypes.byref(ldt), ctypes.byref(ta)),
                   "rrf_get_reflectors")
        f64 = torch.float64
        V = self._copy_out(v.value, ldv.value, m, k, f64)
        T = self._copy_out(t.value, ldt.value, ldt.value, k, f64)
        tau = self._copy_out(ta.value, max(k, 1), k, 1, f64)[:, 0]
        torch.cuda.synchronize(self.device)
        return V, T, tau

    def panel_qr(self, Y):
        """Panel Householder QR + T of a column-major m x b tensor."""
        ldy = _check_colmajor(Y, "Y")
        m, b = Y.shape
        V = _alloc_colmajor(m, b, m, self.dtype, self.device)
        T = _alloc_colmajor(b, b, b, self.dtype, self.device)
        tau = _torch().empty(b, dtype=self.dtype, device=self.device)
        _abi.check(self.lib.rrf_panel_qr(
            self.handle, ctypes.c_void_p(Y.data_ptr()), m, b, ldy,
            ctypes.c_void_p(V.data_ptr()), m, ctypes.c_void_p(T.data_ptr()), b,
            ctypes.c_void_p(tau.data_ptr())), "rrf_panel_qr")
        return V, T, tau

    def apply_block_reflector(self, V, T, X, trans=True):
        """X <- (I - V T V^T)^T X (trans) or (I - V T V^T) X, in place."""
        ldv = _check_colmajor(V, "V")
        ldt = _check_colmajor(T, "T")
        ldx = _check_colmajor(X, "X")
        m, b = V.shape
        _abi.check(self.lib.rrf_apply_block_reflector(
            self.handle, 1 if trans else 0, ctypes.c_void_p(V.data_ptr()), ldv,
            ctypes.c_void_p(T.data_ptr()), ldt, b, ctypes.c_void_p(X.data_ptr()),
            X.shape[0], X.shape[1], ldx), "rrf_apply_block_reflector")
        return X

    def subspace_map(self, Q_new, Q_old, M):
        """GaLore subspace map: Q_new^T (Q_old M) as a new column-major tensor."""
        for t, name in ((Q_new, "Q_new"), (Q_old, "Q_old"), (M, "M")):
            if t.dtype != self.dtype:
                raise TypeError(f"{name}'s dtype differs from the plan's")
        ldqn = _check_colmajor(Q_new, "Q_new")
        ldqo = _check_colmajor(Q_old, "Q_old")
        ldm = _check_colmajor(M, "M")
        m, r_new = Q_new.shape
        if Q_old.shape[0] != m or M.shape[0] != Q_old.shape[1]:
            raise ValueError("shapes do not chain: Q_new m x r1, Q_old m x r0, M r0 x n")
        r_old, n = Q_old.shape[1], M.shape[1]
        out = _alloc_colmajor(r_new, n, max(r_new, 1), self.dtype, self.device)
        _abi.check(self.lib.rrf_subspace_map(
            self.handle, ctypes.c_void_p(Q_new.data_ptr()), ldqn, r_new,
            ctypes.c_void_p(Q_old.data_ptr()), ldqo, r_old,
            ctypes.c_void_p(M.data_ptr()), ldm, m, n,
            ctypes.c_void_p(out.data_ptr()), max(r_new, 1)), "rrf_subspace_map")
        return out


def workspace_size(dtype, m_max, n_max, block_b_max=64, k_max=0):
    """Device bytes a plan with these maxima needs (rrf_workspace_size)."""
    out = ctypes.c_size_t()
    _abi.check(_abi.load().rrf_workspace_size(_dtype_code(dtype), int(m_max), int(n_max),
                                              int(block_b_max), int(k_max),
                                              ctypes.byref(out)),
               "rrf_workspace_size")
    return out.value


def run(A, tol, block_b, seed, k_max=0, stop_mode=RRF_STOP_TRAILING, power=0):
    """One-shot range finder: (Q, B, k) with ||A - Q B||_F <= tol ||A||_F
    (spectral mode: the estimated spectral norm of the residual <= tol
    ||A||_F)."""
    A = colmajor(A)
    m, n = A.shape
    with Plan(A.dtype, max(m, 1), max(n, 1), block_b, k_max,
              device=A.device) as p:
        p.set_stop_mode(stop_mode)
        p.set_power_iterations(power)
        return p.run(A, tol, block_b, seed)


def sketch(dtype, seed, n, col0, ncols, device="cuda", stream=None):
    """Columns [col0, col0 + ncols) of the RRF-NORMAL-v1 sketch (n rows)."""
    torch = _torch()
    out = _alloc_colmajor(n, ncols, max(n, 1), dtype, device)
    if n and ncols:
        _abi.check(_abi.load().rrf_sketch(
            _dtype_code(dtype), int(seed) & 0xFFFFFFFFFFFFFFFF, n, col0, ncols,
            ctypes.c_void_p(out.data_ptr()), max(n, 1),
            _stream_handle(stream)), "rrf_sketch")
    return out
