"""Write the stored expected values under tests/golden/.

Every value written here comes from ``oracle/`` run on ``workloads/`` inputs;
nothing comes from the GPU path.

    python tests/golden/make_golden.py rng        # normal_v1.json (seconds)
    python tests/golden/make_golden.py configs    # oracle_configs.json (long:
                                                  # full-size oracle runs)
    python tests/golden/make_golden.py configs --only square_fp64_16384
"""

import argparse
import json
import math
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import hbarrf, normal_v1  # noqa: E402
import workloads as W  # noqa: E402


def write_rng():
    cases = []
    for seed, n, col0, ncols in [(0, 9, 0, 2), (2001, 33, 5, 3),
                                 (2**64 - 1, 4, 1000, 1), (77, 64, 63, 2)]:
        a = normal_v1(seed, n, col0, ncols)
        cases.append({"seed": seed, "n": n, "col0": col0, "ncols": ncols,
                      "hex": [float(x).hex() for x in a.T.ravel()]})
    with open(os.path.join(HERE, "normal_v1.json"), "w") as f:
        json.dump({"written_by": "tests/golden/make_golden.py rng",
                   "spec": "RRF-NORMAL-v1 (oracle/normal_v1.py)",
                   "cases": cases}, f, indent=1)


def residual_rel(A, Q, B):
    """||A - Q B||_F / ||A||_F in float64, blocked over columns."""
    num = 0.0
    for c0 in range(0, A.shape[1], 1024):
        R = A[:, c0:c0 + 1024].astype(np.float64) - Q @ B[:, c0:c0 + 1024]
        num += float(np.einsum("ij,ij->", R, R))
    den = float(np.einsum("ij,ij->", A.astype(np.float64), A.astype(np.float64)))
    return math.sqrt(num / den)


def orth_err(Q):
    k = Q.shape[1]
    return float(np.linalg.norm(Q.T @ Q - np.eye(k)))


def write_configs(only):
    path = os.path.join(HERE, "oracle_configs.json")
    out = {}
    if os.path.exists(path):
        with open(path) as f:
            out = json.load(f).get("configs", {})
    names = W.CONFIGS + W.GAP_INPUTS
    if only:
        names = [x for x in names if x in only]
    for name in names:
        w = W.WORKLOADS[name]
        t0 = time.time()
        A = W.build_matrix(w)
        t1 = time.time()
        r = hbarrf(A, w.tol, w.block_b, w.sketch_seed, dtype=w.np_dtype)
        t2 = time.time()
        tr = r.trace
        margins = [e / r.sigma2 if r.sigma2 > 0 else None for _, e, _ in tr]
        out[name] = {
            "m": w.m, "n": w.n, "dtype": w.dtype, "block_b": w.block_b,
            "tol": w.tol, "matrix_seed": w.matrix_seed,
            "sketch_seed": w.sketch_seed, "k": r.k, "blocks": len(tr),
            "E0": r.E0, "sigma2": r.sigma2,
            "E_trail_over_sigma2_last2": margins[-2:],
            "E_sub_over_sigma2_last2": [s / r.sigma2 for _, _, s in tr[-2:]],
            "residual_rel": residual_rel(A, r.Q, r.B),
            "orth_fro": orth_err(r.Q),
            "oracle_seconds": t2 - t1, "build_seconds": t1 - t0,
            "numpy": np.__version__,
        }
        print(name, json.dumps(out[name]), flush=True)
        with open(path, "w") as f:
            json.dump({"written_by": "tests/golden/make_golden.py configs",
                       "configs": out}, f, indent=1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("what", choices=["rng", "configs"])
    ap.add_argument("--only", nargs="*", default=None)
    a = ap.parse_args()
    if a.what == "rng":
        write_rng()
    else:
        write_configs(a.only)


if __name__ == "__main__":
    main()
