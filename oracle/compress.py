"""Offline key compression, Algorithm 1 (Sec. III-A, III-C), the plain way.

TEST INFRASTRUCTURE ONLY (like the rest of this package): nothing in the
product path imports it.  Everything is fp64 numpy; each function follows
one step of the method in the paper's order.

  centered(X)               subtract the column means (the CKA definition
                            works on centred representations, Sec. III-A)
  linear_cka(X, Y)          ||Y^T X||_F^2 / (||X^T X||_F ||Y^T Y||_F) on
                            centred X, Y (Sec. III-A)
  head_similarity(A, h, d)  S[i][j] = CKA between the activations of head i
                            and head j: columns i*d .. i*d+d-1 of A (Sec. III-C)
  linkage_distance(D,A,B)   average linkage: mean of D over member pairs
  cluster_heads(S, K)       agglomerative clustering of the heads into K
                            groups (Alg. 1, ClusterHeads)
  energy(W)                 sum of squared singular values = ||W||_F^2
  init_ranks_by_energy      r_i = round(r E_i / E)  (Sec. III-C equation)
  greedy_cost               Delta E_i / alpha_i of lowering group i's rank
  greedy_adjust             lower the rank with the smallest Delta E_i / alpha_i
                            until the budget holds (Sec. III-C)
  group_decompose           per-group truncated SVD, L = U S^1/2, R = S^1/2 V^T
                            (Sec. III-A)
  objective                 sum_i ||W_i - L_i R_i||_F^2 + lam (r - sum_i r_i)
  compress(W, S, r, Ks)     Algorithm 1: the candidate K with the smallest
                            objective

Readings (the paper leaves these open; the same readings are listed with the
design notes):
  * Clustering: average linkage on the distance 1 - S_ij (the paper names
    agglomerative clustering only); on equal distances the pair whose
    smallest head ids are lexicographically smallest merges first.  Groups
    are numbered by their smallest head id, heads inside a group ascending.
  * W's columns of head h are h*d_h .. h*d_h + d_h - 1; a group's W_i takes
    its heads' columns in ascending head order.
  * round() is round-half-up; each r_i is then clipped to [1, min(m, h_i d_h)].
  * The greedy step removes one rank at a time from the group with the
    smallest sigma_{i, r_i}^2 / alpha_i (the energy lost by dropping the last
    kept singular value, per unit of the budget it frees); equal costs go to
    the lower group id; a group keeps at least rank 1.  It runs until
    sum r_i alpha_i <= 4 r / h AND sum r_i <= r: the second condition is the
    problem statement's sum r_i = r, which rounding can overshoot.
  * A candidate set is given by the caller (the paper leaves it unstated);
    on equal objectives the smaller K wins.
  * CKA of a representation with zero variance is taken as 0.
"""

from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------- Sec. III-A
def centered(X: np.ndarray) -> np.ndarray:
    X = np.asarray(X, dtype=np.float64)
    return X - X.mean(axis=0, keepdims=True)


def linear_cka(X: np.ndarray, Y: np.ndarray) -> float:
    """Linear CKA of two representations with the same rows (centred here)."""
    Xc, Yc = centered(X), centered(Y)
    num = np.linalg.norm(Yc.T @ Xc, "fro") ** 2
    den = np.linalg.norm(Xc.T @ Xc, "fro") * np.linalg.norm(Yc.T @ Yc, "fro")
    return float(num / den) if den > 0 else 0.0


def head_similarity(acts: np.ndarray, num_heads: int, head_dim: int) -> np.ndarray:
    """S[i][j] = CKA(activations of head i, activations of head j)."""
    acts = np.asarray(acts, dtype=np.float64)
    assert acts.shape[1] == num_heads * head_dim
    S = np.zeros((num_heads, num_heads))
    for i in range(num_heads):
        for j in range(num_heads):
            S[i, j] = linear_cka(acts[:, i * head_dim:(i + 1) * head_dim],
                                 acts[:, j * head_dim:(j + 1) * head_dim])
    return S


# ---------------------------------------------------------------- Sec. III-C
def linkage_distance(D: np.ndarray, A: Sequence[int], B: Sequence[int]) -> float:
    """Average linkage: the mean of D over the member pairs of clusters A, B."""
    return float(np.mean([D[i, j] for i in A for j in B]))


def cluster_heads(S: np.ndarray, K: int) -> List[List[int]]:
    """Average-linkage agglomerative clustering on 1 - S down to K groups."""
    h = S.shape[0]
    assert 1 <= K <= h
    D = 1.0 - np.asarray(S, dtype=np.float64)
    clusters: List[List[int]] = [[i] for i in range(h)]
    while len(clusters) > K:
        best = None
        for a in range(len(clusters)):
            for b in range(a + 1, len(clusters)):
                key = (linkage_distance(D, clusters[a], clusters[b]), min(clusters[a]), min(clusters[b]))
                if best is None or key < best[0]:
                    best = (key, a, b)
        _, a, b = best
        merged = sorted(clusters[a] + clusters[b])
        clusters = [c for k, c in enumerate(clusters) if k not in (a, b)] + [merged]
        clusters.sort(key=min)
    return clusters


def group_of_head(groups: Sequence[Sequence[int]], num_heads: int) -> List[int]:
    g = [-1] * num_heads
    for gi, members in enumerate(groups):
        for h in members:
            g[h] = gi
    return g


def group_matrices(W: np.ndarray, groups: Sequence[Sequence[int]], head_dim: int) -> List[np.ndarray]:
    """W_i: the columns of group i's heads, in ascending head order."""
    W = np.asarray(W, dtype=np.float64)
    return [np.concatenate([W[:, h * head_dim:(h + 1) * head_dim] for h in sorted(members)], axis=1)
            for members in groups]


def energy(W: np.ndarray) -> float:
    """Sum of squared singular values, which is the squared Frobenius norm."""
    return float(np.sum(np.asarray(W, dtype=np.float64) ** 2))


def init_ranks_by_energy(W_groups: Sequence[np.ndarray], W: np.ndarray, r: int) -> List[int]:
    """r_i = round(r E_i / E), round half up, clipped to [1, min(m, h_i d_h)]."""
    E = energy(W)
    ranks = []
    for Wi in W_groups:
        ri = int(np.floor(r * energy(Wi) / E + 0.5))
        ranks.append(max(1, min(ri, min(Wi.shape))))
    return ranks


def budget_holds(ranks: Sequence[int], heads: Sequence[int], r: int) -> bool:
    """sum_i r_i alpha_i <= 4 r / h, compared exactly."""
    h = sum(heads)
    return sum(Fraction(ri * hi, h) for ri, hi in zip(ranks, heads)) <= Fraction(4 * r, h)


def greedy_cost(sigma_i: np.ndarray, r_i: int, h_i: int, h: int) -> float:
    """Delta E_i / alpha_i: the energy of group i's last kept singular value
    per unit of the budget its removal frees (alpha_i = h_i / h)."""
    return float(sigma_i[r_i - 1] ** 2 / (h_i / h))


def greedy_adjust(ranks: Sequence[int], sigmas: Sequence[np.ndarray], heads: Sequence[int],
                  r: int) -> List[int]:
    """Drop one rank at a time from the group with the smallest
    sigma_{i,r_i}^2 / alpha_i until the budget holds and sum r_i <= r.
    sigmas[i] holds group i's singular values in descending order."""
    h = sum(heads)
    ranks = list(ranks)
    while not (budget_holds(ranks, heads, r) and sum(ranks) <= r):
        best = None
        for i, (ri, hi) in enumerate(zip(ranks, heads)):
            if ri <= 1:
                continue
            cost = greedy_cost(sigmas[i], ri, hi, h)
            if best is None or cost < best[0]:
                best = (cost, i)
        if best is None:                                  # every group is at rank 1
            break
        ranks[best[1]] -= 1
    return ranks


def group_decompose(Wi: np.ndarray, ri: int) -> Tuple[np.ndarray, np.ndarray]:
    """Rank-r_i truncated SVD: L = U_r S_r^1/2, R = S_r^1/2 V_r^T."""
    U, s, Vt = np.linalg.svd(np.asarray(Wi, dtype=np.float64), full_matrices=False)
    sq = np.sqrt(s[:ri])
    return U[:, :ri] * sq[None, :], sq[:, None] * Vt[:ri]


def reconstruction_error(W_groups, factors) -> float:
    return float(sum(np.sum((Wi - L @ R) ** 2) for Wi, (L, R) in zip(W_groups, factors)))


def objective(W_groups, factors, ranks: Sequence[int], r: int, lam: float = 1.0) -> float:
    """sum_i ||W_i - L_i R_i||_F^2 + lam (r - sum_i r_i)."""
    return reconstruction_error(W_groups, factors) + lam * (r - sum(ranks))


def compress(W: np.ndarray, S: np.ndarray, r: int, candidates: Sequence[int], head_dim: int,
             lam: float = 1.0) -> dict:
    """Algorithm 1: cluster, allocate ranks, decompose, score every candidate
    K; return the best one (smallest objective, then smallest K)."""
    W = np.asarray(W, dtype=np.float64)
    num_heads = S.shape[0]
    assert W.shape[1] == num_heads * head_dim
    results = []
    for K in candidates:
        groups = cluster_heads(S, K)
        heads = [len(g) for g in groups]
        Wg = group_matrices(W, groups, head_dim)
        ranks0 = init_ranks_by_energy(Wg, W, r)
        sig = [np.linalg.svd(Wi, compute_uv=False) for Wi in Wg]
        ranks = greedy_adjust(ranks0, sig, heads, r)
        factors = [group_decompose(Wi, ri) for Wi, ri in zip(Wg, ranks)]
        results.append(dict(K=K, groups=groups, heads=heads, init_ranks=ranks0, ranks=ranks,
                            factors=factors, error=reconstruction_error(Wg, factors),
                            objective=objective(Wg, factors, ranks, r, lam)))
    best = min(results, key=lambda d: (d["objective"], d["K"]))
    return dict(best=best, all=results)
