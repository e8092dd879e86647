"""The seeded input generators: determinism and prescribed structure."""

import numpy as np

import workloads as W


def test_deterministic_and_fortran_ordered():
    w = W.scaled("galore_fp32_4096x4096", 200, 150)
    a = W.build_matrix(w)
    b = W.build_matrix(w)
    assert a.dtype == np.float32 and a.flags.f_contiguous
    assert np.array_equal(a, b)


def test_orthofactor_spectrum_is_exact():
    w = W.WORKLOADS["tiny_fp64_500x300"]
    A = W.build_matrix(w)
    s = np.linalg.svd(A, compute_uv=False)
    ref = 10.0 ** (-np.arange(300) / 30.0)
    assert np.max(np.abs(s - ref)) < 1e-13


def test_exact_rank_inputs():
    w = W.WORKLOADS["gap_exact_rank48_fp64"]
    s = np.linalg.svd(W.build_matrix(w), compute_uv=False)
    assert s[47] > 0.4 and s[48] < 1e-14


def test_lowrank_noise_structure():
    w = W.scaled("tall_fp64_131072x2048", 3000, 256)
    A = W.build_matrix(w)
    s = np.linalg.svd(A, compute_uv=False)
    # Signal rank 200 (scaled: min(200, m, n)) above a ~1e-10 noise floor.
    assert s[199] > 1e-9 and s[201] < 1e-9


def test_config_table():
    assert len(W.CONFIGS) == 5
    for name in W.CONFIGS + W.GAP_INPUTS:
        w = W.WORKLOADS[name]
        assert w.block_b >= 1 and 0 < w.tol < 1
