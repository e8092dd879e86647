"""CPU oracle for the Householder blocked adaptive randomized range finder.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and its
Python binding) may import, call or link anything in this package.  Only the
test suite, the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle is a plain, slow implementation written from the paper
(Penke & Herten, "A GPU-Accelerated Blocked Adaptive Randomized Range Finder
Based on an Implicit Householder QR Decomposition"):

* ``normal_v1``   -- the counter-based Gaussian sketch RRF-NORMAL-v1 that both
                     the oracle and the GPU path implement from its definition
                     (the paper only asks for standard Gaussian entries,
                     Alg. 2, sketch step).
* ``hbarrf``      -- Alg. 2 step by step, with unblocked Householder
                     reflections (geqr2 semantics), in float64; optionally
                     with the spectral-norm stopping test and the power
                     iterations the conclusion proposes.
* ``spectral_estimate`` -- the estimate of the spectral norm of the rows not
                     yet in B that the spectral stopping test uses.
* ``stability``   -- the Sec. 6 stability experiment (Fig. 3) in fp32:
                     Alg. 2 against block Gram-Schmidt (Alg. 1) with and
                     without reorthogonalisation (``python -m oracle.stability``).
* ``subspace_map`` -- the GaLore subspace-consistency map of Sec. 7,
                     Q_{t+1}^T Q_t M_t, in float64.

Every function cites the passage it follows.  Pins against independent facts
(LAPACK, SVD, closed forms, invariants) live in ``tests/test_oracle_*.py``.
"""

from .normal_v1 import normal_v1, philox4x64_10_py
from .range_finder import (
    hbarrf,
    householder_vector,
    apply_reflector,
    apply_block_transpose,
    geqr2,
    larft,
    org2r,
    frob2,
    spectral_estimate,
)
from .subspace import subspace_map

__all__ = [
    "normal_v1",
    "philox4x64_10_py",
    "hbarrf",
    "householder_vector",
    "apply_reflector",
    "apply_block_transpose",
    "geqr2",
    "larft",
    "org2r",
    "frob2",
    "spectral_estimate",
    "subspace_map",
]
