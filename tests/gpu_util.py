"""Helpers for the GPU tests (host-side metrics in float64)."""

import math
import sys

import numpy as np


def say(msg):
    """Name the case before a GPU step (visible even if the step faults)."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def to_dev(a):
    import torch
    import paper_2608_28941_amd as rrf
    t = torch.from_numpy(np.asfortranarray(a)).to("cuda")
    return rrf.colmajor(t)


def to_host(t):
    import torch
    torch.cuda.synchronize()
    return np.asfortranarray(t.cpu().numpy())


def orth_err(Q):
    Q = np.asarray(Q, dtype=np.float64)
    return float(np.linalg.norm(Q.T @ Q - np.eye(Q.shape[1])))


def rel_residual(A, Q, B):
    A = np.asarray(A, dtype=np.float64)
    Q = np.asarray(Q, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    return float(np.linalg.norm(A - Q @ B) / np.linalg.norm(A))


def projector_distance(Q, Qo):
    """||Q Q^T - Qo Qo^T||_2 for equal-size bases, as ||Q - Qo (Qo^T Q)||_2
    (the sine of the largest principal angle; no cancellation)."""
    Q = np.asarray(Q, dtype=np.float64)
    Qo = np.asarray(Qo, dtype=np.float64)
    return float(np.linalg.norm(Q - Qo @ (Qo.T @ Q), 2))


def residual_bound(res_oracle, dtype):
    """Spec bar: within 1.05x the oracle's residual; where both sit at
    roundoff (exact-rank inputs) 100 unit roundoffs of the dtype."""
    u = np.finfo(dtype).eps / 2
    return max(1.05 * res_oracle, 100 * u)


ORTH_TOL = {np.dtype(np.float64): 1e-12, np.dtype(np.float32): 1e-5}
PROJ_TOL = {np.dtype(np.float64): 1e-8, np.dtype(np.float32): 1e-3}


def gpu_metrics_torch(A_dev, Q_dev, B_dev):
    """Orthogonality and residual of device results, in float64 on the GPU
    (for full-size inputs too large to move to the host cheaply)."""
    import torch
    Q = Q_dev.to(torch.float64)
    B = B_dev.to(torch.float64)
    A = A_dev.to(torch.float64)
    k = Q.shape[1]
    G = Q.t().contiguous() @ Q
    G -= torch.eye(k, dtype=torch.float64, device=Q.device)
    orth = float(torch.linalg.norm(G))
    num = 0.0
    step = 2048
    for c0 in range(0, A.shape[1], step):
        R = A[:, c0:c0 + step] - Q @ B[:, c0:c0 + step]
        num += float((R * R).sum())
    den = float((A * A).sum())
    return orth, math.sqrt(num / den)
