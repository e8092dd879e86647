"""Stage parity on the GPU: each row of the method against the oracle.

* sketch  -- bit-exact against oracle.normal_v1 (integer-decided bits and a
             fixed sequence of correctly rounded binary64 operations);
* panel   -- V, tau, T against the oracle's geqr2 / larft on the same panel,
             for the three panel algorithms (column by column, from the
             Gram matrix with one exchange per sweep, and tall-skinny QR with
             Householder reconstruction);
* larfb   -- block reflector application against the oracle's reflector-by-
             reflector application (both directions; binary64 X of at most 64
             columns takes the one-launch thin kernel of the look-ahead).
Tolerances for the floating-point stages are relative to the problem scale
and the panel's conditioning (stated per test).
"""

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import say, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2608_28941_amd as rrf  # noqa: E402


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("seed,n,col0,ncols", [
    (0, 1, 0, 1), (2001, 300, 0, 16), (7, 4097, 63, 65), (2**64 - 1, 33, 5, 3),
    (123456789, 100003, 1000, 100)])
def test_sketch_bit_exact(dtype, seed, n, col0, ncols):
    say(f"sketch dtype={np.dtype(dtype).name} seed={seed} n={n} col0={col0} ncols={ncols}")
    tdt = torch.float64 if dtype == np.float64 else torch.float32
    got = to_host(rrf.sketch(tdt, seed, n, col0, ncols))
    want = oracle.normal_v1(seed, n, col0, ncols, dtype=dtype)
    assert got.dtype == want.dtype
    bad = np.count_nonzero(np.ascontiguousarray(got).view(np.uint8)
                           != np.ascontiguousarray(want).view(np.uint8))
    assert bad == 0, f"{bad} bytes differ"


PANEL_CASES = [(500, 16, 1), (64, 64, 2), (1000, 37, 3), (4096, 32, 4),
               (16384, 64, 5), (300, 5, 6), (131072, 32, 7)]


@pytest.mark.parametrize("mode", ["grid", "gram", "tsqr"])
@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("m,b,seed", PANEL_CASES)
def test_panel_qr_matches_oracle(monkeypatch, mode, dtype, m, b, seed):
    # The panel algorithm is chosen when the plan is created.
    monkeypatch.setenv("RRF_PANEL", mode)
    say(f"panel mode={mode} dtype={np.dtype(dtype).name} m={m} b={b}")
    Y = W.random_graded(m, b, dtype, seed, decay=1e-2)
    V_o, tau_o = oracle.geqr2(Y.astype(np.float64))
    T_o = oracle.larft(V_o, tau_o)
    with rrf.Plan(torch.float64 if dtype == np.float64 else torch.float32,
                  m, max(b, 1), b) as p:
        V, T, tau = p.panel_qr(to_dev(Y))
        V, T, tau = to_host(V), to_host(T), to_host(tau)
    # Householder QR is backward stable: with cond(Y) = 100 the reflectors
    # agree to ~cond * u.
    tol = 100 * 100 * np.finfo(dtype).eps
    assert np.max(np.abs(tau - tau_o)) < tol
    assert np.max(np.abs(V - V_o)) < tol * max(1.0, np.max(np.abs(V_o)))
    assert np.max(np.abs(np.triu(T) - np.triu(T_o))) < tol * np.max(np.abs(T_o))
    assert np.all(np.tril(T, -1) == 0)
    assert np.all(np.triu(V, 1) == 0) and np.all(np.diag(V) == 1)


def _rank_deficient(m, b, r, seed):
    g = np.random.default_rng(seed)
    return np.asfortranarray(g.standard_normal((m, r)) @ g.standard_normal((r, b)))


@pytest.mark.parametrize("mode", ["grid", "gram", "tsqr"])
@pytest.mark.parametrize("case", ["graded1e-8", "graded1e-13", "rank12of32", "zero_cols"])
def test_panel_qr_hard_panels(monkeypatch, mode, case):
    """Ill-conditioned and rank-deficient panels: whatever route computes
    the inner products (the Gram route downdates norms and must re-form F
    when they cancel), the reflectors stay orthogonal and Q^T Y is upper
    triangular to binary64 roundoff.  Q = I - V T V^T is orthogonal iff
    M = T^T (V^T V) T - T - T^T vanishes (Q^T Q - I = V M V^T)."""
    monkeypatch.setenv("RRF_PANEL", mode)
    if case == "graded1e-8":
        Y = W.random_graded(4096, 64, np.float64, 11, decay=1e-8)
    elif case == "graded1e-13":
        Y = W.random_graded(16384, 32, np.float64, 12, decay=1e-13)
    elif case == "rank12of32":
        Y = _rank_deficient(2000, 32, 12, 13)
    else:
        Y = W.random_graded(3000, 48, np.float64, 14, decay=1e-3)
        Y[:, [5, 17, 40]] = 0.0
    m, b = Y.shape
    say(f"hard panel mode={mode} case={case} m={m} b={b}")
    with rrf.Plan(torch.float64, m, b, b) as p:
        V, T, tau = p.panel_qr(to_dev(Y))
        V, T, tau = to_host(V), to_host(T), to_host(tau)
    assert np.all(np.isfinite(V)) and np.all(np.isfinite(T))
    assert np.all(np.triu(V, 1) == 0) and np.all(np.diag(V) == 1)
    G = V.T @ V
    M = T.T @ G @ T - T - T.T
    assert np.linalg.norm(M) * np.linalg.norm(V, 2) ** 2 < 1e-12
    R = Y - V @ (T.T @ (V.T @ Y))           # Q^T Y
    ny = np.linalg.norm(Y)
    assert np.linalg.norm(R[b:, :]) <= 1e-13 * ny
    assert np.linalg.norm(np.tril(R[:b, :], -1)) <= 1e-13 * ny
    if case == "zero_cols":
        # A zero column below the diagonal gives tau = 0 only if nothing
        # remains of it after the previous reflectors; the property checks
        # above are what must hold.
        assert np.all(tau >= 0) and np.all(tau <= 2)


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("trans", [True, False])
@pytest.mark.parametrize("m,n,b,seed", [(200, 100, 16, 1), (777, 333, 45, 2),
                                        (4096, 1000, 64, 3), (64, 7, 8, 4),
                                        (16384, 64, 64, 5), (3001, 48, 32, 6),
                                        (60000, 37, 50, 7)])
def test_block_reflector_matches_oracle(dtype, trans, m, n, b, seed):
    say(f"larfb dtype={np.dtype(dtype).name} trans={trans} m={m} n={n} b={b}")
    Y = W.random_graded(m, b, np.float64, seed, decay=1e-2)
    V_o, tau_o = oracle.geqr2(Y)
    T_o = oracle.larft(V_o, tau_o)
    X = W.random_dense(m, n, dtype, seed + 10)
    ref = X.astype(np.float64).copy(order="F")
    if trans:
        oracle.apply_block_transpose(ref, V_o, tau_o)
    else:
        for j in reversed(range(b)):
            oracle.apply_reflector(ref[j:, :], V_o[j:, j], tau_o[j])
    tdt = torch.float64 if dtype == np.float64 else torch.float32
    with rrf.Plan(tdt, m, n, 64) as p:
        Xd = to_dev(X)
        p.apply_block_reflector(to_dev(V_o.astype(dtype)), to_dev(T_o.astype(dtype)),
                                Xd, trans=trans)
        got = to_host(Xd)
    scale = np.linalg.norm(X.astype(np.float64), 2)
    tol = 50 * np.sqrt(b) * np.finfo(dtype).eps * scale
    assert np.max(np.abs(got - ref)) < tol
