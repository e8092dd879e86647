"""Pins for the Alg. 2 oracle against facts that do not come from it.

Each step is checked against something independent:
* panel QR (V, tau)   -- LAPACK dgeqrf on the same panel (same dlarfg
                         convention), and the invariants tau ||v||^2 = 2 and
                         Q^T Y upper triangular;
* T factor            -- LAPACK dgeqrt's T, and I - V T V^T = H_0 ... H_{b-1}
                         formed explicitly;
* block update        -- LAPACK dgemqrt (side L, trans T) on the same (V, T, B);
* stopping quantity   -- brute-force ||A - Q B||_F^2, and the Frobenius
                         identity ||A||^2 - ||B||^2 (Sec. 3);
* whole result        -- the plain definition through Theorem 3.1:
                         Q = numpy qr(A Omega[:, :k]).Q, B = Q^T A, and k the
                         smallest block multiple meeting the tolerance;
* optimality          -- Eckart--Young on an SVD (Sec. 1);
* exact rank          -- k = ceil(r / b) b and roundoff-level residual;
* termination         -- at most ceil(k_cap / b) blocks (Sec. 4).
Planted mistakes in a copy of the oracle (wrong sign, Q_i instead of Q_i^T,
dropped tau, wrong rows in E, transposed T) must each fail one of these.
"""

import math

import numpy as np
import pytest
import scipy.linalg.lapack as lapack

import oracle
from oracle import (hbarrf, householder_vector, apply_reflector, geqr2, larft,
                    org2r, frob2, normal_v1)
import oracle.range_finder as H
import workloads as W

U64 = np.finfo(np.float64).eps


def _panel(m, b, seed, cond=1e2):
    return W.random_graded(m, b, np.float64, seed, decay=1.0 / cond)


# ----------------------------------------------------------------------------
# Pin functions (return an error measure; tests compare with a bound).  The
# planted-mistake test re-runs them against a mutated oracle.
# ----------------------------------------------------------------------------

def pin_geqr2_vs_lapack(m=120, b=16, seed=3):
    Y = _panel(m, b, seed)
    V, tau = geqr2(Y)
    qr, tau_l, _, info = lapack.dgeqrf(Y)
    assert info == 0
    V_l = np.tril(qr[:, :b], -1) + np.eye(m, b)
    return max(np.max(np.abs(V - V_l)), np.max(np.abs(tau - tau_l)))


def pin_larft_vs_lapack(m=90, b=12, seed=4):
    Y = _panel(m, b, seed)
    V, tau = geqr2(Y)
    T = larft(V, tau)
    _, T_l, info = lapack.dgeqrt(b, Y)
    assert info == 0
    return np.max(np.abs(np.triu(T) - np.triu(T_l)))


def pin_block_update_vs_lapack(m=80, n=50, b=10, seed=5):
    Y = _panel(m, b, seed)
    X = W.random_dense(m, n, np.float64, seed + 1)
    V, tau = geqr2(Y)
    T = larft(V, tau)
    mine = np.array(X, order="F")
    oracle.apply_block_transpose(mine, V, tau)
    ref, info = lapack.dgemqrt(V, T, X, side="L", trans="T")
    assert info == 0
    return np.max(np.abs(mine - ref))


def pin_definition(m=300, n=200, b=16, tol=1e-3, seed=6):
    """Theorem 3.1: Q equals the Householder QR of A Omega[:, :k]."""
    w = W.scaled("tiny_fp64_500x300", m, n, block_b=b, tol=tol)
    A = W.build_matrix(w)
    r = hbarrf(A, tol, b, seed)
    Om = normal_v1(seed, n, 0, r.k)
    Y = A @ Om
    Qd = np.linalg.qr(Y)[0]
    sv = np.linalg.svd(Y, compute_uv=False)
    cond = sv[0] / sv[-1]
    errQ = np.max(np.abs(r.Q - Qd)) / (cond * U64 * 1e3)
    errB = np.max(np.abs(r.B - Qd.T @ A)) / (cond * U64 * 1e3)
    # k: the smallest multiple of b whose basis meets the tolerance.
    nA = np.linalg.norm(A)
    Om_all = normal_v1(seed, n, 0, min(m, n))
    k_def = None
    for kk in range(b, min(m, n) + b, b):
        kk = min(kk, min(m, n))
        Qk = np.linalg.qr(A @ Om_all[:, :kk])[0]
        if np.linalg.norm(A - Qk @ (Qk.T @ A)) <= tol * nA:
            k_def = kk
            break
    return max(errQ, errB), r.k, k_def


def pin_E_bruteforce(m=150, n=120, b=8, tol=1e-2, seed=7):
    A = W.random_graded(m, n, np.float64, seed, decay=1e-6)
    r = hbarrf(A, tol, b, seed)
    worst = 0.0
    for (kk, e_trail, e_sub) in r.trace:
        Q = r.Q[:, :kk]
        res2 = np.linalg.norm(A - Q @ (Q.T @ A)) ** 2
        worst = max(worst, abs(e_trail - res2) / r.E0)
    return worst


# ----------------------------------------------------------------------------
# The pins on the real oracle
# ----------------------------------------------------------------------------

def test_householder_vector_convention():
    x = np.array([3.0, 4.0])
    v, tau, beta = householder_vector(x)
    assert beta == -5.0 and v[0] == 1.0
    Hx = x - tau * v * (v @ x)
    assert np.allclose(Hx, [beta, 0.0], atol=1e-15)
    # Negative alpha flips beta; -0.0 counts as positive.
    assert householder_vector(np.array([-3.0, 4.0]))[2] == 5.0
    assert householder_vector(np.array([-0.0, 1.0]))[2] == -1.0
    # x[1:] = 0 gives the identity.
    v, tau, beta = householder_vector(np.array([-2.0, 0.0, 0.0]))
    assert tau == 0.0 and beta == -2.0 and list(v) == [1.0, 0.0, 0.0]


@pytest.mark.parametrize("m,b,seed", [(120, 16, 3), (37, 5, 11), (64, 64, 12),
                                      (500, 32, 13)])
def test_geqr2_matches_lapack(m, b, seed):
    assert pin_geqr2_vs_lapack(m, b, seed) < 1e-12


def test_geqr2_invariants():
    Y = _panel(200, 24, 21, cond=1e6)
    V, tau = geqr2(Y)
    # tau ||v||^2 = 2 for every non-trivial reflector.
    for j in range(24):
        assert abs(tau[j] * (V[:, j] @ V[:, j]) - 2.0) < 1e-13
        assert 1.0 <= tau[j] <= 2.0
    # Q^T Y is upper triangular (lower part at roundoff).
    X = np.array(Y, order="F")
    oracle.apply_block_transpose(X, V, tau)
    assert np.max(np.abs(np.tril(X, -1))) < 1e-13 * np.linalg.norm(Y)


def test_geqr2_zero_column_gives_identity_reflector():
    Y = _panel(40, 6, 22)
    Y[:, 2] = 0.0
    Y[1:, 0] = 0.0            # already triangular first column
    V, tau = geqr2(Y)
    qr, tau_l, _, _ = lapack.dgeqrf(Y)
    assert tau[0] == 0.0 and tau_l[0] == 0.0
    assert np.allclose(tau, tau_l, atol=1e-14)
    assert np.allclose(V, np.tril(qr[:, :6], -1) + np.eye(40, 6), atol=1e-13)


@pytest.mark.parametrize("m,b,seed", [(90, 12, 4), (64, 16, 5), (33, 1, 6)])
def test_larft_matches_lapack(m, b, seed):
    assert pin_larft_vs_lapack(m, b, seed) < 1e-12


def test_larft_explicit_product():
    Y = _panel(20, 5, 8)
    V, tau = geqr2(Y)
    T = larft(V, tau)
    P = np.eye(20)
    for j in range(5):
        P = P @ (np.eye(20) - tau[j] * np.outer(V[:, j], V[:, j]))
    assert np.max(np.abs(P - (np.eye(20) - V @ T @ V.T))) < 1e-14
    assert np.allclose(P.T @ P, np.eye(20), atol=1e-14)


@pytest.mark.parametrize("m,n,b,seed", [(80, 50, 10, 5), (64, 7, 16, 9)])
def test_block_update_matches_lapack(m, n, b, seed):
    assert pin_block_update_vs_lapack(m, n, b, seed) < 1e-12


def test_block_update_preserves_frobenius_norm():
    Y = _panel(100, 8, 31)
    X = W.random_dense(100, 40, np.float64, 32)
    V, tau = geqr2(Y)
    Z = np.array(X, order="F")
    oracle.apply_block_transpose(Z, V, tau)
    assert abs(np.linalg.norm(Z) - np.linalg.norm(X)) < 1e-13 * np.linalg.norm(X)


def test_org2r_matches_lapack():
    Y = _panel(70, 9, 33)
    V, tau = geqr2(Y)
    Q = org2r(V, tau)
    qr, tau_l, _, _ = lapack.dgeqrf(Y)
    Q_l, _, info = lapack.dorgqr(qr, tau_l)
    assert info == 0
    assert np.max(np.abs(Q - Q_l[:, :9])) < 1e-13


def test_whole_result_is_the_plain_definition():
    err, k, k_def = pin_definition()
    assert err < 1.0
    assert k == k_def


@pytest.mark.parametrize("name,m,n,b,tol", [
    ("tiny_fp64_500x300", 500, 300, 16, 1e-4),
    ("galore_fp32_4096x4096", 256, 256, 32, 1e-2),
    ("mlp_fp32_4096x11008", 160, 300, 16, 1e-3),
    ("tall_fp64_131072x2048", 900, 64, 8, 1e-8),
])
def test_qr_of_sketch_and_B(name, m, n, b, tol):
    w = W.scaled(name, m, n, block_b=b, tol=tol)
    A = W.build_matrix(w)
    r = hbarrf(A, tol, b, w.sketch_seed, dtype=w.np_dtype)
    assert r.k % b == 0 or r.k == min(m, n)
    Om = normal_v1(w.sketch_seed, n, 0, r.k, dtype=w.np_dtype).astype(np.float64)
    A64 = A.astype(np.float64)
    Y = A64 @ Om
    R = r.Q.T @ Y
    # Theorem 3.1: Q^T A Omega is upper triangular.
    assert np.max(np.abs(np.tril(R, -1))) < 1e-11 * np.linalg.norm(Y)
    # B = Q^T A (Eq. (2)) and Q^T Q = I (Eq. (1)).
    assert np.max(np.abs(r.B - r.Q.T @ A64)) < 1e-13 * np.linalg.norm(A64)
    assert np.linalg.norm(r.Q.T @ r.Q - np.eye(r.k)) < 1e-13
    # The tolerance is met, and the block before did not meet it.
    res = np.linalg.norm(A64 - r.Q @ r.B) / np.linalg.norm(A64)
    assert res <= tol * (1 + 1e-12)
    if r.k >= b:
        Qp = r.Q[:, :r.k - b]
        assert np.linalg.norm(A64 - Qp @ (Qp.T @ A64)) > tol * np.linalg.norm(A64)


def test_E_trail_is_the_residual():
    assert pin_E_bruteforce() < 1e-13


def test_E_sub_is_the_frobenius_identity():
    A = W.random_graded(120, 90, np.float64, 40, decay=1e-3)
    r = hbarrf(A, 1e-2, 8, 40, stop="subtract")
    for (kk, e_trail, e_sub) in r.trace:
        Bk = r.B[:kk]
        assert abs(e_sub - (r.E0 - frob2(Bk))) < 1e-13 * r.E0
        assert abs(e_sub - e_trail) < 1e-12 * r.E0


def test_eckart_young_lower_bounds():
    A = W.random_graded(80, 60, np.float64, 41, decay=1e-5)
    s = np.linalg.svd(A, compute_uv=False)
    for tol in (1e-1, 1e-2, 1e-3):
        r = hbarrf(A, tol, 8, 41)
        res2 = np.linalg.norm(A - r.Q @ r.B, 2)
        resF = np.linalg.norm(A - r.Q @ r.B)
        k = r.k
        if k < len(s):
            assert res2 >= s[k] * (1 - 1e-12)
            assert resF >= math.sqrt(np.sum(s[k:] ** 2)) * (1 - 1e-12)
        assert resF <= tol * np.linalg.norm(A) * (1 + 1e-12)


@pytest.mark.parametrize("dtype,tol,resid", [(np.float64, 1e-10, 1e-13),
                                             (np.float32, 1e-4, 1e-6)])
def test_exact_rank(dtype, tol, resid):
    name = ("gap_exact_rank48_fp64" if dtype == np.float64
            else "gap_exact_rank48_fp32")
    w = W.WORKLOADS[name]
    A = W.build_matrix(w)
    r = hbarrf(A, tol, w.block_b, w.sketch_seed, dtype=dtype)
    assert r.k == 48
    res = np.linalg.norm(A.astype(np.float64) - r.Q @ r.B) / np.linalg.norm(A)
    assert res < resid
    # rank 50 with b = 16 rounds up to 64
    w2 = W.Workload("r50", 200, 150, w.dtype, 16, tol, 77, 78, kind="exact_rank",
                    rank=50, spectrum="exact_rank")
    r2 = hbarrf(W.build_matrix(w2), tol, 16, 78, dtype=dtype)
    assert r2.k == 64


def test_termination_and_caps():
    A = W.random_graded(60, 20, np.float64, 42, decay=1e-2)
    r = hbarrf(A, 0.0, 8, 42)                   # tol 0: runs to k_cap
    assert r.k == 20 and len(r.trace) == 3      # blocks 8, 8, 4 (ragged)
    assert r.trace[-1][1] < 1e-28 * r.E0        # trailing rows numerically 0
    assert r.status == H.STATUS_OK
    r = hbarrf(A, 1e-9, 8, 42, k_max=12)
    assert r.k == 12 and r.status == H.STATUS_WARN_KMAX
    r = hbarrf(A, 1e-9, 64, 42)                 # b > min(m, n): one block
    assert r.k == 20 and len(r.trace) == 1
    At = np.asfortranarray(A.T)                 # wide
    r = hbarrf(At, 0.0, 8, 42)
    assert r.k == 20
    assert np.linalg.norm(r.Q.T @ r.Q - np.eye(20)) < 1e-13


def test_degenerate_inputs():
    Z = np.zeros((30, 20))
    assert hbarrf(Z, 1e-3, 8, 1).k == 0
    A = W.random_dense(30, 20, np.float64, 43)
    assert hbarrf(A, 1.0, 8, 1).k == 0
    assert hbarrf(A, 5.0, 8, 1).k == 0
    r = hbarrf(np.zeros((0, 5)), 1e-3, 4, 1)
    assert r.k == 0 and r.Q.shape == (0, 0)
    A[3, 4] = np.nan
    with pytest.raises(FloatingPointError):
        hbarrf(A, 1e-3, 8, 1)
    with pytest.raises(ValueError):
        hbarrf(np.ones((4, 4)), float("inf"), 2, 1)
    with pytest.raises(ValueError):
        hbarrf(np.ones((4, 4)), -1.0, 2, 1)


def test_orthogonality_levels():
    for name, m, n, b, tol in [("square_fp64_16384", 700, 600, 32, 1e-6),
                               ("tall_fp64_131072x2048", 2000, 128, 16, 1e-8)]:
        w = W.scaled(name, m, n, block_b=b, tol=tol)
        r = hbarrf(W.build_matrix(w), tol, b, w.sketch_seed)
        assert np.linalg.norm(r.Q.T @ r.Q - np.eye(r.k)) < 1e-13


def test_subtract_and_trailing_agree_above_noise_floor():
    A = W.random_graded(200, 160, np.float64, 44, decay=1e-4)
    a = hbarrf(A, 1e-3, 16, 44)
    b = hbarrf(A, 1e-3, 16, 44, stop="subtract")
    assert a.k == b.k
    assert np.array_equal(a.Q, b.Q)


# ----------------------------------------------------------------------------
# Planted mistakes: each one must make at least one pin fail.
# ----------------------------------------------------------------------------

def _wrong_sign(x):
    """beta takes the sign of alpha (not LAPACK's choice)."""
    x = np.asarray(x, dtype=np.float64)
    alpha = float(x[0])
    xi = float(np.linalg.norm(x[1:])) if x.shape[0] > 1 else 0.0
    v = np.zeros_like(x)
    v[0] = 1.0
    if xi == 0.0:
        return v, 0.0, alpha
    nrm = math.hypot(alpha, xi)
    beta = nrm if alpha >= 0.0 else -nrm
    v[1:] = x[1:] / (alpha - beta)
    return v, (beta - alpha) / beta, beta


_orig_hv = H.householder_vector


def _apply_Qi_not_transpose(X, V, tau):
    for j in reversed(range(len(tau))):
        H.apply_reflector(X[j:, :], V[j:, j], tau[j])


def _dropped_tau(X, v, tau):
    _orig_ar(X, v, 1.0 if tau != 0.0 else 0.0)


_orig_ar = H.apply_reflector


def _larft_transposed(V, tau):
    return _orig_larft(V, tau).T


_orig_larft = H.larft


def _frob_off_by_one(X):
    return _orig_frob(X[1:]) if X.shape[0] > 1 else _orig_frob(X)


_orig_frob = H.frob2


def _run_pins():
    """Return True iff every pin passes on the oracle as currently patched."""
    ok = pin_geqr2_vs_lapack() < 1e-12
    ok &= pin_larft_vs_lapack() < 1e-12
    ok &= pin_block_update_vs_lapack() < 1e-12
    err, k, k_def = pin_definition()
    ok &= (err < 1.0) and (k == k_def)
    ok &= pin_E_bruteforce() < 1e-13
    return bool(ok)


@pytest.mark.parametrize("target,replacement", [
    ("householder_vector", _wrong_sign),
    ("apply_block_transpose", _apply_Qi_not_transpose),
    ("apply_reflector", _dropped_tau),
    ("larft", _larft_transposed),
    ("frob2", _frob_off_by_one),
])
def test_planted_mistake_is_caught(monkeypatch, target, replacement):
    assert _run_pins()
    monkeypatch.setattr(H, target, replacement)
    # The test module imported some names directly; patch those too.
    g = globals()
    if target in g:
        monkeypatch.setitem(g, target, replacement)
    if hasattr(oracle, target):
        monkeypatch.setattr(oracle, target, replacement)
    assert not _run_pins()
