"""Alg. 2 of the paper (Householder Blocked Adaptive Randomized Range Finder),
oracle side.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Plain float64 numpy, one Householder reflection at a time.  The readings of
the paper that this file takes (all listed in the design doc as well):

* Tolerance (Eq. (3) and the guarantee of Alg. 2): relative Frobenius,
  sigma = tol * ||A||_F; the loop runs while E > sigma^2.
* Block update (Alg. 2, update step): the block row update applies
  Q_i^T = I - V_i T_i^T V_i^T, as in Theorem 3.1 (A~ = Q_1^T A); the printed
  (I - V T V^T) would apply Q_i and break the theorem's invariant.  Applying
  Q_i^T is the same as applying H_0, H_1, ..., H_{b-1} in that order, which is
  what this file does.
* Stopping quantity: by default E = ||B[k:, :]||_F^2, the squared norm of the
  rows not yet in B -- in exact arithmetic equal to the paper's running
  difference ||A||_F^2 - sum ||B_i||_F^2 (the Frobenius identity quoted in
  Sec. 3).  The paper reports that the running difference cancels near the
  noise floor (Sec. 6) and lists this as open; ``stop="subtract"`` selects
  the paper's literal rule (clamped at 0, as the paper's figure does).
* Ragged shapes: the rank is capped at k_cap = min(m, n, k_max); the last
  block has width min(b, k_cap - k).  The paper assumes divisibility (Sec. 4).
* Householder convention: LAPACK dlarfg (v[0] = 1,
  beta = -sign(alpha) ||x|| with alpha = +-0 counted as positive,
  tau = (beta - alpha) / beta, tau = 0 when x[1:] = 0).
* Precision: inputs (A and the sketch) are first rounded to the working dtype
  of the configuration, then everything is computed in float64.
* Spectral stopping (``stop="spectral"``; the alternative Sec. 3 mentions
  and the conclusion leaves to future work): the spectral norm of the rows
  not yet in B is estimated after each block by ``spectral_estimate`` on the
  next sketch block (its first min(b, 64) columns), and the loop stops once
  the estimate is <= sigma^2 (sigma = tol ||A||_F, as in the other modes).
* Power iterations (``power=q``; the conclusion's proposal for slowly
  decaying spectra, A replaced by (A A^T)^q A): each block's sample is
  (B B^T)^q B Omega_i on the rows not yet in B, with no orthonormalisation
  between the products.
"""

from dataclasses import dataclass, field
import math

import numpy as np

from .normal_v1 import normal_v1

_CHUNK = 256  # columns per temporary in a rank-1 update (bounds memory only)

STATUS_OK = 0
STATUS_WARN_KMAX = 1


def frob2(X):
    """Squared Frobenius norm, float64 sum of squares."""
    X = np.asarray(X, dtype=np.float64)
    if X.size == 0:
        return 0.0
    return float(np.einsum("ij,ij->", X, X))


def householder_vector(x):
    """Reflector H = I - tau v v^T with H x = beta e_1 and v[0] = 1.

    LAPACK dlarfg semantics (reading R8; Householder QR background, Sec. 2,
    compact WY Eq. (4)).  Returns (v, tau, beta).
    """
    x = np.asarray(x, dtype=np.float64)
    alpha = float(x[0])
    xi = float(np.linalg.norm(x[1:])) if x.shape[0] > 1 else 0.0
    v = np.zeros_like(x)
    v[0] = 1.0
    if xi == 0.0:
        return v, 0.0, alpha
    nrm = math.hypot(alpha, xi)
    beta = -nrm if alpha >= 0.0 else nrm
    tau = (beta - alpha) / beta
    v[1:] = x[1:] / (alpha - beta)
    return v, tau, beta


def apply_reflector(X, v, tau):
    """X <- (I - tau v v^T) X, in place (X is a view into a larger array)."""
    if tau == 0.0 or X.shape[0] == 0 or X.shape[1] == 0:
        return
    w = v @ X
    tv = tau * v
    for c0 in range(0, X.shape[1], _CHUNK):
        X[:, c0:c0 + _CHUNK] -= np.outer(tv, w[c0:c0 + _CHUNK])


def geqr2(Y):
    """Unblocked Householder QR of an m x b panel (LAPACK geqr2 semantics).

    The paper factors each sampled panel with geqrt (Alg. 2, qr step); geqrt
    produces the same reflectors as geqr2 plus the T factor (``larft``).
    Returns (V, tau): V is m x b unit lower trapezoidal; R is discarded, as
    the paper does not need it (Sec. 3).
    """
    Y = np.array(Y, dtype=np.float64, order="F", copy=True)
    m, b = Y.shape
    V = np.zeros((m, b), dtype=np.float64, order="F")
    tau = np.zeros(b, dtype=np.float64)
    for j in range(min(m, b)):
        v, t, _ = householder_vector(Y[j:, j])
        V[j:, j] = v
        tau[j] = t
        apply_reflector(Y[j:, j + 1:], v, t)
    return V, tau


def apply_block_transpose(X, V, tau):
    """X <- Q_i^T X = H_{b-1} ... H_1 H_0 X for the reflectors in V's columns.

    Column j of V is zero above row j (V is unit lower trapezoidal), so H_j
    only touches rows j.. of X.  Alg. 2's block update, read as Q_i^T (R1).
    """
    for j in range(len(tau)):
        apply_reflector(X[j:, :], V[j:, j], tau[j])


def larft(V, tau):
    """Upper triangular T with H_0 H_1 ... H_{b-1} = I - V T V^T.

    Compact WY representation (Eq. (4)); forward, columnwise recursion:
    T[j, j] = tau_j and T[:j, j] = -tau_j T[:j, :j] (V[:, :j]^T v_j).
    """
    V = np.asarray(V, dtype=np.float64)
    b = len(tau)
    T = np.zeros((b, b), dtype=np.float64)
    for j in range(b):
        T[j, j] = tau[j]
        if j:
            T[:j, j] = -tau[j] * (T[:j, :j] @ (V[:, :j].T @ V[:, j]))
    return T


def org2r(V, tau):
    """Explicit Q = H_0 H_1 ... H_{k-1} [I_k; 0] (LAPACK org2r semantics).

    The paper leaves Q implicit as a product of block reflectors (Sec. 4,
    storage scheme); the explicit m x k basis of Eq. (1) is its first k
    columns.  Reflectors are applied from the last to the first.
    """
    V = np.asarray(V, dtype=np.float64)
    m, k = V.shape
    Q = np.zeros((m, k), dtype=np.float64, order="F")
    Q[:k, :k] = np.eye(k)
    for j in range(k - 1, -1, -1):
        apply_reflector(Q[j:, j:], V[j:, j], tau[j])
    return Q


def spectral_estimate(Bt, Om):
    """Estimate of ||Bt||_2^2 from a Gaussian block Om: the largest squared
    norm of Bt^T x over unit x in span(Bt Om), i.e. ||P Bt||_2^2 with P the
    orthogonal projector onto that span (one step of randomized subspace
    iteration; a lower bound of ||Bt||_2^2, exact when rank(Bt) <= the
    block width).  The span is taken from an SVD of Y = Bt Om, dropping
    directions below the roundoff of Y."""
    Bt = np.asarray(Bt, dtype=np.float64)
    if Bt.size == 0 or Om.shape[1] == 0:
        return 0.0
    Y = Bt @ Om
    U, sv, _ = np.linalg.svd(Y, full_matrices=False)
    if sv.size == 0 or sv[0] == 0.0:
        return 0.0
    r = int(np.count_nonzero(sv > sv[0] * max(Y.shape) * np.finfo(np.float64).eps))
    return float(np.linalg.norm(U[:, :r].T @ Bt, 2) ** 2)


@dataclass
class HbarrfResult:
    k: int
    Q: np.ndarray          # m x k, orthonormal columns
    B: np.ndarray          # k x n, B = Q^T A
    V: np.ndarray          # m x k, Householder vectors (unit lower trapezoidal)
    tau: np.ndarray        # k
    T_blocks: list         # T_i per block (b_i x b_i, upper triangular)
    trace: list            # (k after the block, E_trail, E_sub) per block
    E0: float              # ||A||_F^2
    sigma2: float          # (tol ||A||_F)^2
    status: int = STATUS_OK
    extras: dict = field(default_factory=dict)


def hbarrf(A, tol, block_b, seed, k_max=0, dtype=None, stop="trailing", power=0):
    """Alg. 2: blocked adaptive range finder on an implicit Householder QR.

    A        m x n input (its values are used as given; pass A already rounded
             to the working dtype)
    tol      relative Frobenius tolerance, 0 <= tol < inf
    block_b  block size b >= 1
    seed     sketch seed (RRF-NORMAL-v1, domain 0)
    k_max    rank cap; 0 means min(m, n)  (also the fixed-rank mode of Sec. 6)
    dtype    working dtype of the sketch (float32 sketches are the float64
             sketch rounded to nearest-even); default A's dtype
    stop     "trailing" (default), "subtract" (the paper's running
             difference) or "spectral" (estimated spectral norm of the rows
             not yet in B, ``spectral_estimate``)
    power    power iterations per block sample (0: Alg. 2 as printed)
    """
    A = np.asarray(A)
    if A.ndim != 2:
        raise ValueError("A must be a matrix")
    dtype = np.dtype(A.dtype if dtype is None else dtype)
    if dtype not in (np.dtype(np.float32), np.dtype(np.float64)):
        raise ValueError("dtype must be float32 or float64")
    if not (math.isfinite(tol) and tol >= 0.0):
        raise ValueError("tol must be finite and >= 0")
    if block_b < 1 or k_max < 0:
        raise ValueError("block_b must be >= 1 and k_max >= 0")
    if stop not in ("trailing", "subtract", "spectral"):
        raise ValueError("stop must be 'trailing', 'subtract' or 'spectral'")
    if power < 0:
        raise ValueError("power must be >= 0")
    m, n = A.shape

    # Alg. 2 initialisation: E <- ||A||_F^2, B <- A, V <- 0, i <- 0.
    Bw = np.array(A, dtype=np.float64, order="F", copy=True)
    E0 = frob2(Bw)
    if not math.isfinite(E0):
        raise FloatingPointError("A has non-finite entries")
    sigma2 = (tol * tol) * E0
    k_cap = min(m, n) if k_max == 0 else min(m, n, k_max)
    V = np.zeros((m, k_cap), dtype=np.float64, order="F")
    tau = np.zeros(k_cap, dtype=np.float64)
    T_blocks = []
    trace = []
    E_trail = E0
    E_sub = E0
    E_spec = E0      # before any block the test falls back on ||A||_F^2
    k = 0

    def current_E():
        return {"trailing": E_trail, "subtract": E_sub, "spectral": E_spec}[stop]

    # Alg. 2 loop: while E > sigma^2 (and ranks remain, Sec. 4 termination).
    while current_E() > sigma2 and k < k_cap:
        bi = min(block_b, k_cap - k)
        # Fresh Gaussian block: global sketch columns [k, k + bi).
        Om = normal_v1(seed, n, k, bi, dtype=dtype).astype(np.float64)
        # (V_i, T_i) <- qr(B_{i:j} Omega)  -- sample the not-yet-final rows,
        # optionally (B B^T)^q B Omega.
        Y = Bw[k:, :] @ Om
        for _ in range(power):
            Y = Bw[k:, :] @ (Bw[k:, :].T @ Y)
        Vi, ti = geqr2(Y)
        V[k:, k:k + bi] = Vi
        tau[k:k + bi] = ti
        T_blocks.append(larft(Vi, ti))
        # B_{i:j} <- Q_i^T B_{i:j}, one reflector at a time (reading R1).
        apply_block_transpose(Bw[k:, :], Vi, ti)
        # E <- E - ||B_i||_F^2 (paper), and the direct trailing norm.
        E_sub = max(0.0, E_sub - frob2(Bw[k:k + bi, :]))
        E_trail = frob2(Bw[k + bi:, :])
        k += bi
        if stop == "spectral":
            # On the next sketch block's first min(b, 64) columns.
            p = min(block_b, 64, k_cap - k)
            if p > 0:
                On = normal_v1(seed, n, k, p, dtype=dtype).astype(np.float64)
                E_spec = spectral_estimate(Bw[k:, :], On)
            else:
                E_spec = float("nan")
        trace.append((k, E_trail, E_sub) if stop != "spectral"
                     else (k, E_trail, E_sub, E_spec))

    status = STATUS_OK
    # At the cap the spectral estimate is not formed; the Frobenius norm (an
    # upper bound of the spectral norm) decides the warning there.
    E_end = E_trail if stop == "spectral" else current_E()
    if E_end > sigma2 and k == k_cap and k_cap < min(m, n):
        status = STATUS_WARN_KMAX
    Q = org2r(V[:, :k], tau[:k])
    B = np.array(Bw[:k, :], order="F", copy=True)
    return HbarrfResult(k=k, Q=Q, B=B, V=np.array(V[:, :k], order="F"),
                        tau=tau[:k].copy(), T_blocks=T_blocks, trace=trace,
                        E0=E0, sigma2=sigma2, status=status)
