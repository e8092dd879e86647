"""GaLore subspace-consistency map (Sec. 7 of the paper), oracle side.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

With an adaptive range finder the basis of a layer's low-rank optimizer
state changes from one training step to the next (Q_t, m x r_t, then
Q_{t+1}, m x r_{t+1}, possibly of another rank).  Sec. 7 carries a state
M_t (r_t x n) expressed in the old basis into the new one by the linear map
M_t -> Q_{t+1}^T Q_t M_t.  This file writes that definition out in float64,
with numpy's matrix product as the step: first the state back in the
ambient space (Q_t M_t, m x n), then its coordinates in the new basis.
"""

import numpy as np


def subspace_map(Q_new, Q_old, M):
    """Q_new^T (Q_old M) in float64 (Sec. 7)."""
    Q_new = np.asarray(Q_new, dtype=np.float64)
    Q_old = np.asarray(Q_old, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    if Q_new.shape[0] != Q_old.shape[0] or Q_old.shape[1] != M.shape[0]:
        raise ValueError("shapes do not chain: Q_new m x r1, Q_old m x r0, M r0 x n")
    ambient = Q_old @ M
    return Q_new.T @ ambient
