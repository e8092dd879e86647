"""Pins for the oracle's Gaussian sketch (RRF-NORMAL-v1).

What fixes each part, independently of the oracle's own code:
* raw bits     -- a Philox4x64-10 written from the SC'11 definition
                  (``philox4x64_10_py``) against numpy's Philox (an independent
                  library implementation); this also fixes the counter layout;
* ln, sin, cos -- the C library (math.log / math.sin / math.cos) to a few ulp;
* Box--Muller  -- the row formula rebuilt from the words and libm, and the
                  distribution (moments, Kolmogorov--Smirnov against N(0, 1));
* placement    -- prefix and block-split invariance, which the definition
                  implies (column g of the n x inf sketch does not depend on n
                  or on the block size);
* regression   -- stored hex values written by tests/golden/make_golden.py.
"""

import json
import math
import os

import numpy as np
import pytest
import scipy.stats

from oracle import normal_v1, philox4x64_10_py
from oracle.normal_v1 import (_cos_sin_2pi, _ln, philox_words, normal_column,
                              TWO_M53)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("seed,domain,column", [
    (0, 0, 0), (5, 0, 0), (5, 0, 1), (2**64 - 1, 0, 7), (12345, 3, 2**20 + 3),
    (0xDEADBEEFCAFEF00D, 1, 99)])
def test_philox_words_match_definition(seed, domain, column):
    w = philox_words(seed, domain, column, 5)
    for q in range(5):
        ref = philox4x64_10_py((q, column, 0, 0), (seed, domain))
        assert tuple(int(x) for x in w[q]) == ref


def test_philox_definition_is_not_trivial():
    # Different counters / keys give different words (guards a degenerate
    # implementation that ignores an input).
    a = philox4x64_10_py((0, 0, 0, 0), (1, 0))
    assert a != philox4x64_10_py((1, 0, 0, 0), (1, 0))
    assert a != philox4x64_10_py((0, 1, 0, 0), (1, 0))
    assert a != philox4x64_10_py((0, 0, 0, 0), (2, 0))
    assert a != philox4x64_10_py((0, 0, 0, 0), (1, 1))


def _ulp(x):
    return math.ulp(abs(x)) if x != 0 else math.ulp(0.0)


def test_ln_accuracy_against_libm():
    rng = np.random.default_rng(1)
    u = np.concatenate([
        rng.random(20000) + TWO_M53,
        np.array([TWO_M53, 2 * TWO_M53, 0.5, 1.0, 1.0 - TWO_M53,
                  float.fromhex("0x1.6a09e667f3bcdp-1"),
                  float.fromhex("0x1.6a09e667f3bccp-1"),
                  float.fromhex("0x1.6a09e667f3bcep-1"), 0.25, 0.75]),
        np.exp(-rng.random(5000) * 36.0)])
    u = np.clip(u, TWO_M53, 1.0)
    got = _ln(u)
    for x, g in zip(u, got):
        ref = math.log(x)
        assert abs(g - ref) <= 4 * _ulp(ref) + 1e-300, (x, g, ref)
    assert _ln(np.array([1.0]))[0] == 0.0


def test_cos_sin_accuracy_against_libm():
    rng = np.random.default_rng(2)
    u = np.concatenate([rng.random(20000),
                        np.array([0.0, 0.25, 0.5, 0.75, 1.0 - TWO_M53,
                                  0.125, 0.375, 0.625, 0.875])])
    c, s = _cos_sin_2pi(u)
    ref_c = np.cos(2.0 * math.pi * u)
    ref_s = np.sin(2.0 * math.pi * u)
    # Argument reduction by quadrant is exact; the only argument error is the
    # rounding of pi/2, so an absolute bound of a few ulp(1) holds.
    assert np.max(np.abs(c - ref_c)) < 2e-15
    assert np.max(np.abs(s - ref_s)) < 2e-15
    assert np.allclose(c * c + s * s, 1.0, atol=1e-15, rtol=0)
    # Exact quadrant points.
    c0, s0 = _cos_sin_2pi(np.array([0.0, 0.25, 0.5, 0.75]))
    assert list(c0) == [1.0, 0.0, -1.0, 0.0] or np.allclose(
        c0, [1, 0, -1, 0], atol=1e-16)
    assert np.allclose(s0, [0, 1, 0, -1], atol=1e-16)


def test_row_formula_from_words():
    """Rows 4q..4q+3 from (w0,w1) and (w2,w3), rebuilt with libm."""
    seed, n, col = 77, 37, 5
    z = normal_column(seed, n, col)
    for q in range((n + 3) // 4):
        w = philox4x64_10_py((q, col, 0, 0), (seed, 0))
        vals = []
        for a, b in ((w[0], w[1]), (w[2], w[3])):
            u1 = ((a >> 11) + 1) * 2.0 ** -53
            u2 = (b >> 11) * 2.0 ** -53
            r = math.sqrt(-2.0 * math.log(u1))
            vals += [r * math.cos(2 * math.pi * u2),
                     r * math.sin(2 * math.pi * u2)]
        for t in range(4):
            row = 4 * q + t
            if row < n:
                assert abs(z[row] - vals[t]) <= 1e-14 * max(1.0, abs(vals[t]))


def test_distribution_is_standard_normal():
    x = normal_v1(2024, 4096, 0, 256).ravel()   # 2^20 draws
    nsamp = x.size
    assert abs(x.mean()) < 4.0 / math.sqrt(nsamp)
    assert abs(x.var() - 1.0) < 4.0 * math.sqrt(2.0 / nsamp)
    assert abs(np.mean(x ** 4) - 3.0) < 4.0 * math.sqrt(96.0 / nsamp)
    assert scipy.stats.kstest(x, "norm").pvalue > 1e-3
    # Neighbouring rows / columns are uncorrelated.
    X = normal_v1(2025, 4096, 0, 64)
    C = np.corrcoef(X.T)
    assert np.max(np.abs(C - np.eye(64))) < 0.08
    assert abs(np.corrcoef(X[0::2, 0], X[1::2, 0])[0, 1]) < 0.08


def test_placement_invariances():
    seed = 31337
    big = normal_v1(seed, 301, 0, 12)
    small = normal_v1(seed, 150, 0, 12)
    assert np.array_equal(big[:150], small)            # independent of n
    parts = np.hstack([normal_v1(seed, 301, 0, 5), normal_v1(seed, 301, 5, 7)])
    assert np.array_equal(parts, big)                  # independent of b
    assert not np.array_equal(big[:, 0], big[:, 1])
    assert not np.array_equal(normal_v1(seed + 1, 301, 0, 1)[:, 0], big[:, 0])
    assert not np.array_equal(normal_v1(seed, 301, 0, 1, domain=1)[:, 0],
                              big[:, 0])


def test_float32_is_rounded_float64():
    a64 = normal_v1(9, 257, 3, 9)
    a32 = normal_v1(9, 257, 3, 9, dtype=np.float32)
    assert a32.dtype == np.float32
    assert np.array_equal(a32, a64.astype(np.float32))


def test_stored_values_unchanged():
    with open(os.path.join(GOLDEN, "normal_v1.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        got = normal_v1(case["seed"], case["n"], case["col0"], case["ncols"])
        want = np.array([float.fromhex(h) for h in case["hex"]]).reshape(
            case["ncols"], case["n"]).T
        assert np.array_equal(got, want)
