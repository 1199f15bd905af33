"""Value calibration refinement (Sec. III-D), the plain way.

TEST INFRASTRUCTURE ONLY (like the rest of this package).  fp64 numpy.

The value projection W (m x n, acting on row vectors: x W) is factored by a
truncated SVD into L_v (m x r, producing the cached latent z = x L_v) and
R_v (r x n, the up-projection), as in Sec. III-A.  The calibration error on
N calibration inputs X (N x m, one token a row) is

    eps = ||X L_v R_v - X W||_F^2.

Reading of the closed forms.  The paper states the error and the two
updates with the weight acting on calibration columns from the left; in the
row convention used everywhere else (Sec. III-A) that is the transposed
problem, so its first update (of the factor that does not meet the data
directly) is the update of R_v and its second the update of L_v.  With the
Gram matrix G = X^T X:

    R_v <- (L_v^T G L_v)^{-1} L_v^T G W          (sets d eps / d R_v to 0)
    L_v <- W R_v^T (R_v R_v^T)^{-1}              (sets d eps / d L_v to 0
                                                  whenever G is nonsingular)

Each update is an exact minimiser of eps over its factor (the second one
when N >= m and X has full column rank), so eps never increases.
"""

from __future__ import annotations

from typing import Tuple

import numpy as np


def svd_factors(W: np.ndarray, r: int) -> Tuple[np.ndarray, np.ndarray]:
    """L_v = U_r S_r^1/2, R_v = S_r^1/2 V_r^T (Sec. III-A)."""
    U, s, Vt = np.linalg.svd(np.asarray(W, dtype=np.float64), full_matrices=False)
    sq = np.sqrt(s[:r])
    return U[:, :r] * sq[None, :], sq[:, None] * Vt[:r]


def gram(X: np.ndarray) -> np.ndarray:
    X = np.asarray(X, dtype=np.float64)
    return X.T @ X


def calib_error(X: np.ndarray, W: np.ndarray, L: np.ndarray, R: np.ndarray) -> float:
    X = np.asarray(X, dtype=np.float64)
    return float(np.sum((X @ L @ R - X @ W) ** 2))


def update_right(G: np.ndarray, W: np.ndarray, L: np.ndarray) -> np.ndarray:
    """R_v = (L^T G L)^{-1} L^T G W."""
    return np.linalg.solve(L.T @ G @ L, L.T @ G @ W)


def update_left(W: np.ndarray, R: np.ndarray) -> np.ndarray:
    """L_v = W R^T (R R^T)^{-1}, solved as (R R^T) L^T = R W^T."""
    return np.linalg.solve(R @ R.T, R @ W.T).T


def refine(X: np.ndarray, W: np.ndarray, r: int) -> dict:
    """SVD factors, then the R_v update, then the L_v update."""
    L0, R0 = svd_factors(W, r)
    G = gram(X)
    R1 = update_right(G, np.asarray(W, dtype=np.float64), L0)
    L1 = update_left(np.asarray(W, dtype=np.float64), R1)
    return dict(L_svd=L0, R_svd=R0, R_mid=R1, L=L1, R=R1,
                eps_svd=calib_error(X, W, L0, R0), eps_mid=calib_error(X, W, L0, R1),
                eps=calib_error(X, W, L1, R1))
