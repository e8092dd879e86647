"""Seeded synthetic inputs for tests and the benchmark.

This module holds only input generation (random matrices with prescribed
singular-value structure).  It contains none of the range finder's arithmetic
and is the one module shared by the oracle-side tests and the GPU-side tests.

All matrices are built in float64 with numpy's Philox generator and rounded
once to the working dtype.  Noise matrices N have iid N(0, 1) entries scaled by
1/sqrt(max(m, n)).  Factor matrices G have iid N(0, 1) entries scaled by
1/sqrt(their row count).  Seeds are fixed per workload.

The paper uses synthetic random matrices only (Sec. 6: a 1024 x 1024 matrix
with log-spaced singular values and random orthogonal factors; random square
matrices for the runtime study), so no dataset is involved.  The five
workloads below are GaLore-shaped stand-ins (gradient shapes of a LLaMA-7B
layer) plus a large square and a tall-skinny stress case.
"""

from dataclasses import dataclass
import math

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    m: int
    n: int
    dtype: str          # "float32" | "float64"
    block_b: int
    tol: float
    matrix_seed: int
    sketch_seed: int
    kind: str           # construction recipe, see ``build_matrix``
    rank: int = 0       # factor rank (kind "lowrank_noise")
    noise: float = 0.0
    spectrum: str = ""  # name of the singular-value law

    @property
    def np_dtype(self):
        return np.dtype(self.dtype)


# The five configurations of the benchmark (sizes, dtypes, b, tol as stated
# for this build), plus spectral-gap inputs and small scaled copies for tests.
WORKLOADS = {
    "tiny_fp64_500x300": Workload(
        "tiny_fp64_500x300", 500, 300, "float64", 16, 1e-4, 1001, 2001,
        kind="orthofactors", spectrum="pow10_i_over_30"),
    "galore_fp32_4096x4096": Workload(
        "galore_fp32_4096x4096", 4096, 4096, "float32", 32, 1e-2, 1002, 2002,
        kind="lowrank_noise", rank=512, noise=1e-3, spectrum="ipow_m1p5"),
    "mlp_fp32_4096x11008": Workload(
        "mlp_fp32_4096x11008", 4096, 11008, "float32", 64, 1e-3, 1003, 2003,
        kind="lowrank_noise", rank=256, noise=1e-4, spectrum="exp_i_over_40"),
    "square_fp64_16384": Workload(
        "square_fp64_16384", 16384, 16384, "float64", 64, 1e-6, 1004, 2004,
        kind="lowrank_noise", rank=1024, noise=1e-8, spectrum="pow10_i_over_128"),
    "tall_fp64_131072x2048": Workload(
        "tall_fp64_131072x2048", 131072, 2048, "float64", 32, 1e-8, 1005, 2005,
        kind="lowrank_noise", rank=200, noise=1e-10, spectrum="flat50_then_pow10_20"),
    # Spectral-gap inputs (gap at a block boundary).
    "gap_exact_rank48_fp64": Workload(
        "gap_exact_rank48_fp64", 256, 192, "float64", 16, 1e-10, 1101, 2101,
        kind="exact_rank", rank=48, spectrum="exact_rank"),
    "gap_exact_rank48_fp32": Workload(
        "gap_exact_rank48_fp32", 256, 192, "float32", 16, 1e-4, 1102, 2102,
        kind="exact_rank", rank=48, spectrum="exact_rank"),
    "gap_rank128_fp64": Workload(
        "gap_rank128_fp64", 2048, 1024, "float64", 64, 1e-6, 1103, 2103,
        kind="gap_noise", rank=128, noise=1e-13, spectrum="logspace_1_1em2"),
    "gap_rank128_fp32": Workload(
        "gap_rank128_fp32", 2048, 1024, "float32", 64, 1e-3, 1104, 2104,
        kind="gap_noise", rank=128, noise=1e-6, spectrum="logspace_1_1em2"),
}

# Names of the five benchmark configurations, in order.
CONFIGS = [
    "tiny_fp64_500x300",
    "galore_fp32_4096x4096",
    "mlp_fp32_4096x11008",
    "square_fp64_16384",
    "tall_fp64_131072x2048",
]
GAP_INPUTS = [
    "gap_exact_rank48_fp64",
    "gap_exact_rank48_fp32",
    "gap_rank128_fp64",
    "gap_rank128_fp32",
]


def spectrum(name, count):
    """Singular values s_0 .. s_{count-1} of the named law."""
    i = np.arange(count, dtype=np.float64)
    if name == "pow10_i_over_30":
        return 10.0 ** (-i / 30.0)
    if name == "ipow_m1p5":              # s_i = i^-1.5 for i = 1 .. count
        return (i + 1.0) ** -1.5
    if name == "exp_i_over_40":
        return np.exp(-i / 40.0)
    if name == "pow10_i_over_128":
        return 10.0 ** (-i / 128.0)
    if name == "flat50_then_pow10_20":
        return np.where(i < 50, 1.0, 10.0 ** (-(i - 50.0) / 20.0))
    if name == "logspace_1_1em2":
        return np.logspace(0.0, -2.0, count)
    if name == "exact_rank":
        return np.linspace(1.0, 0.5, count)
    raise ValueError(name)


def _rng(seed, stream):
    return np.random.Generator(np.random.Philox(key=[seed, stream]))


def _gaussian_t(rng, m, n):
    """Return an (m, n) Fortran-ordered N(0,1) matrix (generated as its
    C-ordered transpose, so no copy is needed)."""
    return rng.standard_normal((n, m)).T


def build_matrix(w, m=None, n=None):
    """The workload's A (Fortran order, rounded to ``w.dtype``).

    ``m`` / ``n`` override the size (scaled copies for tests keep the recipe
    and the seeds; the spectrum is taken over the smaller factor rank).
    """
    m = w.m if m is None else m
    n = w.n if n is None else n
    if w.kind == "orthofactors":
        # A = X diag(s) Y^T with X, Y the Q factors of Householder QR of
        # Gaussian matrices.
        r = min(m, n)
        X = np.linalg.qr(_gaussian_t(_rng(w.matrix_seed, 1), m, r))[0]
        Y = np.linalg.qr(_gaussian_t(_rng(w.matrix_seed, 2), n, r))[0]
        s = spectrum(w.spectrum, r)
        At = (Y * s) @ X.T                       # n x m, C order == A in F order
        A = At.T
    elif w.kind in ("lowrank_noise", "gap_noise", "exact_rank"):
        r = min(w.rank, m, n)
        G1 = _gaussian_t(_rng(w.matrix_seed, 1), m, r) / math.sqrt(m)
        G2 = _gaussian_t(_rng(w.matrix_seed, 2), n, r) / math.sqrt(n)
        if w.kind == "exact_rank":
            # Orthonormal factors make the rank exact and well conditioned.
            G1 = np.linalg.qr(G1)[0]
            G2 = np.linalg.qr(G2)[0]
        s = spectrum(w.spectrum, r)
        At = np.ascontiguousarray((G2 * s) @ G1.T)   # n x m, C order
        if w.noise:
            Nt = _rng(w.matrix_seed, 3).standard_normal((n, m))
            Nt *= w.noise / math.sqrt(max(m, n))
            At += Nt
            del Nt
        A = At.T
    else:
        raise ValueError(w.kind)
    return np.asfortranarray(A.astype(w.np_dtype, copy=False))


def scaled(name, m, n, block_b=None, tol=None):
    """A smaller copy of a workload with the same recipe and seeds."""
    w = WORKLOADS[name]
    return Workload(f"{w.name}@{m}x{n}", m, n, w.dtype,
                    w.block_b if block_b is None else block_b,
                    w.tol if tol is None else tol,
                    w.matrix_seed, w.sketch_seed, w.kind, w.rank, w.noise,
                    w.spectrum)


def random_dense(m, n, dtype, seed):
    """Plain iid N(0,1) matrix (Fortran order), for stage-level tests."""
    return np.asfortranarray(_gaussian_t(_rng(seed, 7), m, n).astype(dtype))


def random_graded(m, n, dtype, seed, decay=1e-3):
    """m x n matrix with singular values log-spaced from 1 to ``decay``."""
    r = min(m, n)
    U = np.linalg.qr(_gaussian_t(_rng(seed, 8), m, r))[0]
    W = np.linalg.qr(_gaussian_t(_rng(seed, 9), n, r))[0]
    s = np.logspace(0.0, math.log10(decay), r)
    return np.asfortranarray(((U * s) @ W.T).astype(dtype))
