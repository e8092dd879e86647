"""Pins of the oracle's GaLore subspace map (Sec. 7) against facts that do not
use its formula: an unchanged basis leaves the state unchanged, a rotated
basis rotates it, a basis orthogonal to the old one maps it to zero, and
carrying a state through an intermediate basis that contains the old one
equals carrying it directly."""

import numpy as np
import pytest

import oracle


def _orth(m, r, seed):
    rng = np.random.default_rng(seed)
    q, _ = np.linalg.qr(rng.standard_normal((m, r)))
    return q


def test_same_basis_is_identity():
    Q = _orth(300, 24, 1)
    M = np.random.default_rng(2).standard_normal((24, 17))
    assert np.max(np.abs(oracle.subspace_map(Q, Q, M) - M)) < 1e-13


def test_rotated_basis_rotates_the_state():
    Q = _orth(200, 16, 3)
    R = _orth(16, 16, 4)                      # orthogonal 16 x 16
    M = np.random.default_rng(5).standard_normal((16, 9))
    # Q_new = Q R spans the same space: coordinates change by R^T.
    got = oracle.subspace_map(Q @ R, Q, M)
    assert np.max(np.abs(got - R.T @ M)) < 1e-13


def test_orthogonal_basis_maps_to_zero():
    U = _orth(128, 40, 6)
    Q_old, Q_new = U[:, :15], U[:, 15:40]     # complementary columns
    M = np.random.default_rng(7).standard_normal((15, 11))
    got = oracle.subspace_map(Q_new, Q_old, M)
    assert got.shape == (25, 11)
    assert np.max(np.abs(got)) < 1e-13


def test_intermediate_basis_containing_the_old_one():
    U = _orth(150, 30, 8)
    Q1, Q2 = U[:, :10], U[:, :30]             # span(Q1) inside span(Q2)
    Q3 = _orth(150, 12, 9)
    M = np.random.default_rng(10).standard_normal((10, 7))
    two = oracle.subspace_map(Q3, Q2, oracle.subspace_map(Q2, Q1, M))
    one = oracle.subspace_map(Q3, Q1, M)
    assert np.max(np.abs(two - one)) < 1e-12


def test_rank_change_and_shapes():
    Q_old, Q_new = _orth(64, 8, 11), _orth(64, 5, 12)
    M = np.ones((8, 3))
    assert oracle.subspace_map(Q_new, Q_old, M).shape == (5, 3)
    with pytest.raises(ValueError):
        oracle.subspace_map(Q_new, Q_old, np.ones((7, 3)))
