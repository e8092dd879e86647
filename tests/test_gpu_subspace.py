"""GaLore subspace map (Sec. 7) on the GPU against the oracle.

rrf_subspace_map computes Q_new^T (Q_old M) with two dense GEMMs in the
plan's dtype; the oracle computes the same definition in float64 from the
same (rounded) inputs.  Bar: elementwise within 8 sqrt((m + r_old) r_old) u
max|M| (u of the dtype), a dot-product error bound with margin; plus the
cases with an exact answer (unchanged basis, empty old basis)."""

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import say, to_dev, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2608_28941_amd as rrf  # noqa: E402


def _orth(m, r, seed, dtype):
    rng = np.random.default_rng(seed)
    q, _ = np.linalg.qr(rng.standard_normal((m, max(r, 1))))
    return np.asfortranarray(q[:, :r].astype(dtype))


def _tdt(dtype):
    return torch.float64 if dtype == np.float64 else torch.float32


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
@pytest.mark.parametrize("m,r_old,r_new,n", [(300, 24, 17, 50), (4096, 64, 96, 257),
                                             (1000, 7, 1, 3), (512, 32, 32, 1)])
def test_subspace_map_matches_oracle(dtype, m, r_old, r_new, n):
    say(f"subspace_map dtype={np.dtype(dtype).name} m={m} r_old={r_old} r_new={r_new} n={n}")
    Q_old = _orth(m, r_old, 1 + m, dtype)
    Q_new = _orth(m, r_new, 2 + m, dtype)
    M = np.asfortranarray(np.random.default_rng(3).standard_normal((r_old, n)).astype(dtype))
    ref = oracle.subspace_map(Q_new, Q_old, M)
    with rrf.Plan(_tdt(dtype), m, max(n, 1), 64) as p:
        got = to_host(p.subspace_map(to_dev(Q_new), to_dev(Q_old), to_dev(M)))
    assert got.shape == (r_new, n)
    u = np.finfo(dtype).eps / 2
    tol = 8 * np.sqrt((m + r_old) * r_old) * u * np.max(np.abs(M))
    assert np.max(np.abs(got - ref)) <= tol


@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_subspace_map_exact_cases(dtype):
    m, r, n = 777, 40, 33
    Q = _orth(m, r, 5, dtype)
    M = np.asfortranarray(np.random.default_rng(6).standard_normal((r, n)).astype(dtype))
    with rrf.Plan(_tdt(dtype), m, n, 64) as p:
        same = to_host(p.subspace_map(to_dev(Q), to_dev(Q), to_dev(M)))
        empty = to_host(p.subspace_map(to_dev(Q), to_dev(np.zeros((m, 0), dtype)),
                                       to_dev(np.zeros((0, n), dtype))))
    u = np.finfo(dtype).eps / 2
    # Q^T Q = I up to the orthonormality of the rounded Q.
    qtq = Q.astype(np.float64).T @ Q.astype(np.float64)
    bound = (np.max(np.abs(qtq - np.eye(r))) * r + 8 * np.sqrt((m + r) * r) * u) * np.max(np.abs(M))
    assert np.max(np.abs(same - M)) <= bound
    assert empty.shape == (r, n) and not np.any(empty)


def test_subspace_map_between_range_finder_bases():
    # Two consecutive "gradients" of a GaLore-shaped layer: bases of
    # different rank from rrf_run, a state carried from one to the other.
    w = W.scaled("galore_fp32_4096x4096", 512, 384)
    A0 = W.build_matrix(w).astype(np.float64)
    A1 = A0 + 1e-3 * np.random.default_rng(7).standard_normal(A0.shape) / np.sqrt(512)
    with rrf.Plan(torch.float64, 512, 384, 32) as p:
        Q0, _, k0 = p.run(to_dev(np.asfortranarray(A0)), 1e-2, 32, 11)
        Q0 = to_host(Q0)
        Q1, _, k1 = p.run(to_dev(np.asfortranarray(A1)), 5e-3, 32, 12)
        Q1 = to_host(Q1)
        M = np.asfortranarray(np.random.default_rng(8).standard_normal((k0, 64)))
        got = to_host(p.subspace_map(to_dev(Q1), to_dev(Q0), to_dev(M)))
    say(f"subspace_map between bases k0={k0} k1={k1}")
    ref = oracle.subspace_map(Q1, Q0, M)
    assert got.shape == (k1, 64)
    assert np.max(np.abs(got - ref)) <= 8 * np.sqrt((512 + k0) * k0) * 2**-53 * np.max(np.abs(M))
