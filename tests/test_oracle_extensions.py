"""Pins for the oracle's extensions of Alg. 2 that the conclusion proposes:
spectral-norm stopping (``stop="spectral"``, ``spectral_estimate``) and power
iterations (``power=q``).

Each is checked against facts that do not come from the oracle's formula:
* ``spectral_estimate``  -- never above ||Bt||_2^2 (numpy's 2-norm); equal
                            to it when rank(Bt) <= the block width or when all
                            singular values are equal; within 0.1 % of it on a
                            fast-decaying spectrum;
* spectral stopping      -- on a fast-decaying spectrum (estimate accurate) k
                            is the smallest block multiple whose true spectral
                            residual ||A - Q B||_2 meets sigma; never more
                            columns than the Frobenius rule;
* power iterations       -- power = 0 is Alg. 2 itself; each block's new basis
                            columns span P (A A^T P)^q A Omega_i, with P the
                            projector onto the complement of the earlier
                            columns, formed with explicit projectors and no
                            Householder step; exact rank still gives k = r;
                            a slowly decaying spectrum is approximated better.
Planted mistakes (wrong normalisation, the wrong rows of B, powers on all
rows) must each fail one of these.
"""

import numpy as np
import pytest

import oracle
import oracle.range_finder as H
import workloads as W

U64 = np.finfo(np.float64).eps


def _with_spectrum(m, n, s, seed):
    g = np.random.default_rng(seed)
    U = np.linalg.qr(g.standard_normal((m, len(s))))[0]
    Vt = np.linalg.qr(g.standard_normal((n, len(s))))[0].T
    return np.asfortranarray((U * s) @ Vt)


def _gauss(n, p, seed):
    return np.random.default_rng(seed).standard_normal((n, p))


# ----------------------------------------------------------------------------
# Pin functions (an error measure each; the planted-mistake test re-runs them)
# ----------------------------------------------------------------------------

def pin_estimate_exact_rank(seed=1):
    """rank(Bt) = 12 <= p = 16: the estimate is ||Bt||_2^2."""
    s = np.logspace(0, -3, 12)
    Bt = _with_spectrum(300, 200, s, seed)
    est = H.spectral_estimate(Bt, _gauss(200, 16, seed + 1))
    return abs(est - np.linalg.norm(Bt, 2) ** 2) / s[0] ** 2


def pin_estimate_flat(seed=2):
    """All 150 singular values 0.7: any projection onto a subspace of the
    range has spectral norm 0.7."""
    Bt = _with_spectrum(250, 180, np.full(150, 0.7), seed)
    est = H.spectral_estimate(Bt, _gauss(180, 8, seed + 1))
    return abs(est - 0.49) / 0.49


def pin_estimate_upper_and_close(seed=3):
    """Never above ||Bt||_2^2; within 0.1 % of it on a geometric spectrum
    (ratio 0.79) and within 10 % on a harmonic and a clustered one (one
    power step).  Returns the worst violation (0 when all hold)."""
    worst = 0.0
    for (m, n, p, s, lo) in [(400, 300, 16, 10.0 ** (-np.arange(300) / 10.0), 0.999),
                             (200, 500, 8, 1.0 / (1.0 + np.arange(200)), 0.9),
                             (120, 90, 32, np.ones(90) + np.arange(90) % 3, 0.9)]:
        Bt = _with_spectrum(m, n, s, seed)
        est = H.spectral_estimate(Bt, _gauss(n, p, seed + 7))
        true = np.linalg.norm(Bt, 2) ** 2
        worst = max(worst, max(0.0, est - true * (1 + 1e-12)) / true)
        worst = max(worst, max(0.0, lo * true - est) / true)
    return worst


def pin_spectral_stop(seed=4):
    """Fast decay (estimate accurate): k is the smallest multiple of b with
    ||A - Q_k Q_k^T A||_2 <= sigma (residuals from the oracle's Q at every
    block boundary); returns the number of violations."""
    s = 10.0 ** (-np.arange(150) / 12.0)
    A = _with_spectrum(260, 180, s, seed)
    b, tol, sd = 8, 1e-4, 17
    r = oracle.hbarrf(A, tol, b, sd, stop="spectral")
    sigma = tol * np.linalg.norm(A)
    full = oracle.hbarrf(A, 0.0, b, sd, k_max=r.k + 2 * b)
    res = [np.linalg.norm(A - full.Q[:, :k] @ (full.Q[:, :k].T @ A), 2)
           for k in range(0, r.k + 1, b)]
    bad = int(res[-1] > sigma * (1 + 1e-9))
    bad += sum(int(x <= sigma) for x in res[:-1])
    ft = oracle.hbarrf(A, tol, b, sd)
    bad += int(r.k > ft.k)
    return bad


def pin_power_projectors(q=1, seed=5):
    """Each block's new columns span P (A A^T P)^q A Omega_i (P: projector
    onto the complement of the earlier columns); returns the largest
    projector distance over the blocks."""
    s = 1.0 / np.sqrt(1.0 + np.arange(120))
    A = _with_spectrum(150, 130, s, seed)
    b, sd = 10, 23
    r = oracle.hbarrf(A, 0.0, b, sd, k_max=40, power=q)
    worst = 0.0
    for i in range(0, r.k, b):
        Qp = r.Q[:, :i]
        P = np.eye(A.shape[0]) - Qp @ Qp.T
        Om = oracle.normal_v1(sd, A.shape[1], i, b)
        X = P @ (A @ Om)
        for _ in range(q):
            X = P @ (A @ (A.T @ X))
        Ux = np.linalg.qr(X)[0]
        Qi = r.Q[:, i:i + b]
        worst = max(worst, np.linalg.norm(Qi - Ux @ (Ux.T @ Qi), 2))
    return worst


def _run_pins():
    ok = pin_estimate_exact_rank() < 1e-10
    ok &= pin_estimate_flat() < 1e-10
    ok &= pin_estimate_upper_and_close() == 0.0
    ok &= pin_spectral_stop() == 0
    ok &= pin_power_projectors() < 1e-8
    return bool(ok)


# ----------------------------------------------------------------------------

def test_estimate_exact_when_rank_fits_the_block():
    assert pin_estimate_exact_rank() < 1e-10


def test_estimate_exact_on_a_flat_spectrum():
    assert pin_estimate_flat() < 1e-10


def test_estimate_is_a_lower_bound_and_close_on_fast_decay():
    assert pin_estimate_upper_and_close() == 0.0


def test_estimate_of_zero_and_empty():
    assert H.spectral_estimate(np.zeros((30, 20)), _gauss(20, 4, 1)) == 0.0
    assert H.spectral_estimate(np.zeros((0, 20)), _gauss(20, 4, 1)) == 0.0


def test_spectral_stop_is_the_smallest_meeting_block():
    assert pin_spectral_stop() == 0


def test_spectral_mode_trace_and_degenerate_inputs():
    w = W.scaled("tiny_fp64_500x300", 200, 150, block_b=16, tol=1e-3)
    A = W.build_matrix(w)
    r = oracle.hbarrf(A, w.tol, 16, w.sketch_seed, stop="spectral")
    assert all(len(t) == 4 for t in r.trace)
    # The recorded estimate is what the next test compares with sigma^2.
    for (_, _, _, es) in r.trace[:-1]:
        assert es > r.sigma2
    assert r.trace[-1][3] <= r.sigma2 or r.k == 150
    assert oracle.hbarrf(np.zeros((20, 10)), 1e-3, 4, 1, stop="spectral").k == 0
    assert oracle.hbarrf(A, 1.0, 16, 1, stop="spectral").k == 0
    # Tolerance 0: runs to the cap; the last block has no estimate.
    r0 = oracle.hbarrf(A[:40, :30], 0.0, 8, 1, stop="spectral")
    assert r0.k == 30 and np.isnan(r0.trace[-1][3])


def test_power_zero_is_alg2():
    w = W.scaled("tiny_fp64_500x300", 200, 150, block_b=16, tol=1e-3)
    A = W.build_matrix(w)
    a = oracle.hbarrf(A, w.tol, 16, w.sketch_seed)
    b = oracle.hbarrf(A, w.tol, 16, w.sketch_seed, power=0)
    assert a.k == b.k and np.array_equal(a.Q, b.Q) and np.array_equal(a.B, b.B)


@pytest.mark.parametrize("q", [1, 2])
def test_power_blocks_span_the_deflated_power_subspace(q):
    assert pin_power_projectors(q=q) < 1e-8


def test_power_exact_rank():
    w = W.WORKLOADS["gap_exact_rank48_fp64"]
    A = W.build_matrix(w)
    r = oracle.hbarrf(A, w.tol, w.block_b, w.sketch_seed, power=1)
    assert r.k == 48
    assert np.linalg.norm(A - r.Q @ r.B) / np.linalg.norm(A) < 1e3 * U64
    assert np.linalg.norm(r.Q.T @ r.Q - np.eye(48)) < 1e-13


def test_power_improves_slow_decay():
    # sigma_i = (1 + i)^-1/2: at rank 32 one power step moves the basis
    # much closer to the dominant subspace (Frobenius and spectral residual).
    s = 1.0 / np.sqrt(1.0 + np.arange(300))
    A = _with_spectrum(400, 300, s, 9)
    r0 = oracle.hbarrf(A, 0.0, 16, 31, k_max=32)
    r1 = oracle.hbarrf(A, 0.0, 16, 31, k_max=32, power=1)
    e0 = np.linalg.norm(A - r0.Q @ r0.B, 2)
    e1 = np.linalg.norm(A - r1.Q @ r1.B, 2)
    best = s[32]
    assert e1 < e0
    assert (e1 - best) < 0.5 * (e0 - best)


# ----------------------------------------------------------------------------
# Planted mistakes
# ----------------------------------------------------------------------------

_orig_est = H.spectral_estimate


def _est_no_projection(Bt, Om):
    """||Bt Om||_2^2 / ||Om||_2^2 instead of the projected norm."""
    Y = np.asarray(Bt) @ Om
    return float(np.linalg.norm(Y, 2) ** 2 / np.linalg.norm(Om, 2) ** 2)


def _est_one_row_too_many(Bt, Om):
    return _orig_est(Bt, Om) if Bt.shape[0] < 2 else _orig_est(Bt[:-1], Om) * 0.5


_orig_hbarrf = H.hbarrf


def _hbarrf_power_all_rows(A, tol, block_b, seed, k_max=0, dtype=None, stop="trailing",
                           power=0):
    """Powers taken with the whole matrix A instead of the rows not yet in B
    (no deflation)."""
    if power == 0:
        return _orig_hbarrf(A, tol, block_b, seed, k_max, dtype, stop)
    A = np.asarray(A, dtype=np.float64)
    m, n = A.shape
    k_cap = min(m, n) if k_max == 0 else min(m, n, k_max)
    cols = []
    k = 0
    while k < k_cap:
        bi = min(block_b, k_cap - k)
        X = A @ oracle.normal_v1(seed, n, k, bi)
        for _ in range(power):
            X = A @ (A.T @ X)
        cols.append(X)
        k += bi
    Qf = np.linalg.qr(np.hstack(cols))[0]
    return H.HbarrfResult(k=k, Q=Qf, B=Qf.T @ A, V=None, tau=None, T_blocks=[],
                          trace=[], E0=0.0, sigma2=0.0)


@pytest.mark.parametrize("target,replacement", [
    ("spectral_estimate", _est_no_projection),
    ("spectral_estimate", _est_one_row_too_many),
    ("hbarrf", _hbarrf_power_all_rows),
])
def test_planted_mistake_is_caught(monkeypatch, target, replacement):
    assert _run_pins()
    monkeypatch.setattr(H, target, replacement)
    if hasattr(oracle, target):
        monkeypatch.setattr(oracle, target, replacement)
    assert not _run_pins()
