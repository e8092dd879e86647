"""Stability experiment of Sec. 6 (Fig. 3) on the CPU, in single precision.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``): a CPU experiment that
compares, block by block, three adaptive range finders run in fp32
arithmetic on the same matrix with the same sketch:

* ``hh``          -- Alg. 2 (Householder blocked adaptive randomized range
                     finder): sample the trailing rows, factor the panel with
                     Householder QR (geqrt), apply Q_i^T to the trailing
                     rows (gemqrt), track the paper's E (running difference of
                     panel norms) and the trailing norm.
* ``bcgs``        -- Alg. 1 (block randomized range finder of Martinsson &
                     Voronin) without reorthogonalisation: orthonormalise the
                     sample of the in-place residual with a QR, take
                     B_new = Q_new^T A and subtract Q_new B_new.
* ``bcgs_reorth`` -- Alg. 1 with its reorthogonalisation step,
                     Q_new <- orth((I - Q Q^T) Q_new).

After every block the explicit basis Q (all columns so far) is measured in
float64: the projection residual ||A - Q Q^T A||_2, the loss of
orthogonality ||Q^T Q - I||_2, and the quantity each method tracks for its
stopping test (HH: sqrt(E) with E the running difference clamped at 0, and
the trailing norm; BCGS: ||A - Q B||_2 of the in-place residual).  The test
matrix follows Sec. 6: singular values decaying logarithmically from 1 to
1e-14 with random orthogonal singular vectors, formed in float64 and rounded
to fp32 once.  Library routines serve as the steps (LAPACK sgeqrt / sgemqrt /
sgeqrf through scipy and numpy); no step is blocked or fused beyond the
algorithms' own statements.

Run ``python -m oracle.stability [--n 1024 --b 64]`` for the table.
"""

import argparse
import math

import numpy as np
from scipy.linalg import lapack

from .normal_v1 import normal_v1

F32 = np.float32


def test_matrix(n, seed=3001, smax=0.0, smin=-14.0):
    """A = U diag(s) V^T (n x n), s_i = 10^(smax + i (smin - smax)/(n-1)),
    U, V orthogonal from QR of Gaussian matrices; float64 then rounded to
    fp32 (Sec. 6, stability experiment).  Returns (A32, s)."""
    rng = np.random.Generator(np.random.Philox(seed))
    U, _ = np.linalg.qr(rng.standard_normal((n, n)))
    V, _ = np.linalg.qr(rng.standard_normal((n, n)))
    s = np.logspace(smax, smin, n)
    A = (U * s) @ V.T
    return np.asfortranarray(A.astype(F32)), s


def _measure(A64, Q):
    """(||A - Q Q^T A||_2, ||Q^T Q - I||_2) in float64 for the fp32 basis Q."""
    Q = Q.astype(np.float64)
    R = A64 - Q @ (Q.T @ A64)
    k = Q.shape[1]
    return (float(np.linalg.norm(R, 2)),
            float(np.linalg.norm(Q.T @ Q - np.eye(k), 2)))


def run_hh(A32, b, seed, nblocks=None):
    """Alg. 2 in fp32: per block the sample Y = B[k:, :] Omega_i, geqrt on Y,
    B[k:, :] <- Q_i^T B[k:, :] with gemqrt, then the paper's running E and
    the trailing norm.  Yields per-block records."""
    m, n = A32.shape
    B = np.array(A32, dtype=F32, order="F")
    E = F32(np.sum(B * B, dtype=F32))     # ||A||_F^2, the paper's initial E
    blocks = []                           # (k, V, T) of each block
    k = 0
    A64 = A32.astype(np.float64)
    nb = nblocks or (min(m, n) // b)
    for i in range(nb):
        bi = min(b, min(m, n) - k)
        Om = normal_v1(seed, n, k, bi, dtype=F32)
        Y = (B[k:, :] @ Om).astype(F32)
        V, T, info = lapack.sgeqrt(bi, np.asfortranarray(Y))
        assert info == 0
        Vt = np.tril(V, -1)
        Vt[np.arange(bi), np.arange(bi)] = 1.0
        out, info = lapack.sgemqrt(np.asfortranarray(Vt), T, np.asfortranarray(B[k:, :]),
                                   side="L", trans="T")
        assert info == 0
        B[k:, :] = out
        blocks.append((k, Vt, T))
        panel = B[k:k + bi, :]
        E = F32(E - F32(np.sum(panel * panel, dtype=F32)))
        trail = B[k + bi:, :]
        E_trail = float(np.sum(trail * trail, dtype=F32))
        k += bi
        # Explicit Q = H_0 ... H_{k-1} [I_k; 0]: the block reflectors applied
        # backwards (orgqr semantics), in fp32.
        Q = np.zeros((m, k), dtype=F32, order="F")
        Q[np.arange(k), np.arange(k)] = 1.0
        for (kk, Vb, Tb) in reversed(blocks):
            sub, info = lapack.sgemqrt(np.asfortranarray(Vb), Tb,
                                       np.asfortranarray(Q[kk:, kk:]), side="L", trans="N")
            assert info == 0
            Q[kk:, kk:] = sub
        res, orth = _measure(A64, Q)
        blocks_rec = {"k": k, "residual": res, "orth": orth,
                      "sqrt_E_sub": math.sqrt(max(float(E), 0.0)),
                      "E_sub_negative": bool(float(E) < 0.0),
                      "sqrt_E_trail": math.sqrt(E_trail)}
        yield blocks_rec


def run_bcgs(A32, b, seed, reorth, nblocks=None):
    """Alg. 1 in fp32: the residual A is updated in place; per block
    Q_new = orth(A Omega) [then orth((I - Q Q^T) Q_new)], B_new = Q_new^T A,
    A <- A - Q_new B_new.  Yields per-block records."""
    m, n = A32.shape
    R = np.array(A32, dtype=F32, order="F")
    A64 = A32.astype(np.float64)
    Q = np.zeros((m, 0), dtype=F32)
    k = 0
    nb = nblocks or (min(m, n) // b)
    for i in range(nb):
        bi = min(b, min(m, n) - k)
        Om = normal_v1(seed, n, k, bi, dtype=F32)
        Qn, _ = np.linalg.qr((R @ Om).astype(F32))
        Qn = Qn.astype(F32)
        if reorth and k > 0:
            Qn, _ = np.linalg.qr((Qn - Q @ (Q.T @ Qn)).astype(F32))
            Qn = Qn.astype(F32)
        Q = np.hstack([Q, Qn]).astype(F32)
        Bn = (Qn.T @ R).astype(F32)
        R = (R - Qn @ Bn).astype(F32)
        k += bi
        res, orth = _measure(A64, Q)
        yield {"k": k, "residual": res, "orth": orth,
               "tracked_2norm": float(np.linalg.norm(R.astype(np.float64), 2))}


def experiment(n=1024, b=64, seed=2999, nblocks=None):
    """All three methods on the Sec. 6 matrix; returns (rows, sigma), rows a
    list of per-block dicts keyed by method."""
    A32, s = test_matrix(n)
    sig = np.linalg.svd(A32.astype(np.float64), compute_uv=False)
    hh = list(run_hh(A32, b, seed, nblocks))
    cg = list(run_bcgs(A32, b, seed, False, nblocks))
    cr = list(run_bcgs(A32, b, seed, True, nblocks))
    rows = []
    for i in range(len(hh)):
        k = hh[i]["k"]
        rows.append({"k": k, "hh": hh[i], "bcgs": cg[i], "bcgs_reorth": cr[i],
                     "sigma_prescribed": float(s[k]) if k < n else 0.0,
                     "sigma_actual": float(sig[k]) if k < n else 0.0})
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--n", type=int, default=1024)
    ap.add_argument("--b", type=int, default=64)
    a = ap.parse_args()
    rows = experiment(a.n, a.b)
    print(f"Sec. 6 stability experiment, fp32, {a.n} x {a.n}, b = {a.b}, "
          f"sigma_i = 10^(-14 i/(n-1)); ||.||_2 measured in float64\n")
    print("| k | sigma_k+1 prescribed | actual | HH ||A-QQ^TA|| | BCGS | BCGS+reorth | "
          "HH sqrt(E_sub) | HH trail | BCGS ||A-QB|| | reorth ||A-QB|| | "
          "HH ||Q^TQ-I|| | BCGS | BCGS+reorth |")
    print("|" + "---|" * 13)
    for r in rows:
        hh, cg, cr = r["hh"], r["bcgs"], r["bcgs_reorth"]
        esub = "0 (E < 0)" if hh["E_sub_negative"] else f"{hh['sqrt_E_sub']:.2e}"
        print(f"| {r['k']} | {r['sigma_prescribed']:.2e} | {r['sigma_actual']:.2e} | "
              f"{hh['residual']:.2e} | {cg['residual']:.2e} | {cr['residual']:.2e} | "
              f"{esub} | {hh['sqrt_E_trail']:.2e} | {cg['tracked_2norm']:.2e} | "
              f"{cr['tracked_2norm']:.2e} | {hh['orth']:.2e} | {cg['orth']:.2e} | "
              f"{cr['orth']:.2e} |")


if __name__ == "__main__":
    main()
