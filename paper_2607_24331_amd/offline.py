"""Offline compression of one layer (Algorithm 1 for keys, Sec. III-C; the
calibration refinement for values, Sec. III-D), run once before serving.

The contractions over calibration samples run on the GPU through the
library: the centred Gram of the heads' activations and the CKA head
similarity built from it, and the calibration Gram X^T X.  The steps that
follow are small and run on the host: head clustering and rank allocation
in the library's host code; the per-group SVDs and the two r x r solves of
the value refinement in fp64 LAPACK (numpy), on matrices of the weights'
size rather than the calibration set's.
"""

from __future__ import annotations

from typing import Sequence

import numpy as np
import torch

from .dckv import allocate_ranks, cluster_heads, gram, head_similarity


def key_similarity(acts: torch.Tensor, num_heads: int, head_dim: int) -> torch.Tensor:
    """S [h, h] (fp32, on the GPU): linear CKA between the heads' activations,
    acts [samples, h*d_h] on the GPU (head h in columns h*d_h .. h*d_h+d_h-1)."""
    G = gram(acts, center=True)
    return head_similarity(G, num_heads, head_dim)


def _truncated_factors(U, s, Vt, r):
    sq = np.sqrt(s[:r])
    return U[:, :r] * sq[None, :], sq[:, None] * Vt[:r]


def compress_keys(W, S, r: int, candidates: Sequence[int], head_dim: int, lam: float = 1.0) -> dict:
    """Algorithm 1 for a key projection W [m, h*d_h] (host array) and head
    similarity S [h, h]: for every candidate cluster count K, cluster the
    heads, allocate ranks, factor each group by truncated SVD and score
    sum_i ||W_i - L_i R_i||_F^2 + lam (r - sum_i r_i); return the best K
    (smallest objective, then smallest K) and every candidate's result."""
    W = np.asarray(W, dtype=np.float64)
    S = S.detach().cpu().numpy() if isinstance(S, torch.Tensor) else np.asarray(S)
    h = S.shape[0]
    m = W.shape[0]
    if W.shape[1] != h * head_dim:
        raise ValueError("W must have h * head_dim columns")
    results = []
    for K in candidates:
        gid = cluster_heads(S, K)
        groups = [[hh for hh in range(h) if gid[hh] == g] for g in range(K)]
        Wg = [np.concatenate([W[:, hh * head_dim:(hh + 1) * head_dim] for hh in grp], axis=1)
              for grp in groups]
        svd = [np.linalg.svd(Wi, full_matrices=False) for Wi in Wg]
        energy = [float(np.sum(Wi * Wi)) for Wi in Wg]
        caps = [min(m, Wi.shape[1]) for Wi in Wg]
        init, ranks = allocate_ranks([len(g) for g in groups], energy, float(np.sum(W * W)),
                                     [sv[1] for sv in svd], caps, r)
        factors = [_truncated_factors(U, s, Vt, ri) for (U, s, Vt), ri in zip(svd, ranks)]
        # Eckart-Young: the truncation error is the energy of the dropped singular values
        error = float(sum(np.sum(s[ri:] ** 2) for (_, s, _), ri in zip(svd, ranks)))
        results.append(dict(K=K, groups=groups, heads=[len(g) for g in groups], init_ranks=init,
                            ranks=ranks, factors=factors, error=error,
                            objective=error + lam * (r - sum(ranks))))
    best = min(results, key=lambda d: (d["objective"], d["K"]))
    return dict(best=best, all=results)


def refine_value(W, r: int, X: torch.Tensor) -> dict:
    """Value factors of rank r for W [m, n] (host array), refined on the
    calibration inputs X [samples, m] (GPU): truncated SVD, then
    R_v = (L^T G L)^{-1} L^T G W and L_v = W R_v^T (R_v R_v^T)^{-1} with the
    GPU Gram G = X^T X.  Errors eps = tr((L R - W)^T G (L R - W))."""
    W = np.asarray(W, dtype=np.float64)
    G = gram(X, center=False).double().cpu().numpy()
    U, s, Vt = np.linalg.svd(W, full_matrices=False)
    L0, R0 = _truncated_factors(U, s, Vt, r)
    R1 = np.linalg.solve(L0.T @ G @ L0, L0.T @ G @ W)
    L1 = np.linalg.solve(R1 @ R1.T, R1 @ W.T).T

    def eps(L, R):
        D = L @ R - W
        return float(np.sum(D * (G @ D)))

    return dict(L_svd=L0, R_svd=R0, L=L1, R=R1, gram=G,
                eps_svd=eps(L0, R0), eps_mid=eps(L0, R1), eps=eps(L1, R1))
