"""Pins of the offline key-compression oracle (Algorithm 1; Sec. III-A, III-C)
against what the mathematics and the paper fix: the kernel form of CKA, a
library clustering routine, Eckart-Young, hand-worked greedy steps and the
parameter-count inequality."""

import numpy as np
import pytest
from scipy.cluster.hierarchy import fcluster, linkage
from scipy.spatial.distance import squareform

from oracle import compress as oc
from oracle import params


def _hsic_cka(X, Y):
    # kernel form: tr(K H L H) / sqrt(tr(K H K H) tr(L H L H)), K = X X^T, L = Y Y^T
    N = X.shape[0]
    H = np.eye(N) - np.ones((N, N)) / N
    K, L = X @ X.T, Y @ Y.T
    return np.trace(K @ H @ L @ H) / np.sqrt(np.trace(K @ H @ K @ H) * np.trace(L @ H @ L @ H))


def test_cka_equals_kernel_form():
    g = np.random.default_rng(1)
    for _ in range(5):
        N, dx, dy = 40, int(g.integers(2, 9)), int(g.integers(2, 9))
        X = g.standard_normal((N, dx)) + g.standard_normal(dx)     # nonzero means
        Y = X[:, :min(dx, dy)] @ g.standard_normal((min(dx, dy), dy)) + g.standard_normal((N, dy))
        assert oc.linear_cka(X, Y) == pytest.approx(_hsic_cka(X, Y), rel=1e-12)
        assert oc.linear_cka(X, Y) == pytest.approx(oc.linear_cka(Y, X), rel=1e-12)
        assert 0.0 <= oc.linear_cka(X, Y) <= 1.0 + 1e-12


def test_cka_invariances():
    g = np.random.default_rng(2)
    X = g.standard_normal((64, 8))
    Q, _ = np.linalg.qr(g.standard_normal((8, 8)))
    assert oc.linear_cka(X, X @ Q) == pytest.approx(1.0, abs=1e-12)           # rotation
    assert oc.linear_cka(X, 3.5 * X + 7.0) == pytest.approx(1.0, abs=1e-12)   # scale and shift
    Y = g.standard_normal((4096, 8))
    Z = g.standard_normal((4096, 8))
    assert oc.linear_cka(Y, Z) < 0.05                                         # independent
    assert oc.linear_cka(np.ones((10, 3)), Y[:10, :3]) == 0.0                 # zero variance


def test_head_similarity_planted_pairs():
    g = np.random.default_rng(3)
    N, d = 200, 8
    base = g.standard_normal((N, d))
    Q, _ = np.linalg.qr(g.standard_normal((d, d)))
    acts = np.concatenate([base, base @ Q, g.standard_normal((N, d))], axis=1)
    S = oc.head_similarity(acts, 3, d)
    assert np.allclose(np.diag(S), 1.0)
    assert np.allclose(S, S.T)
    assert S[0, 1] == pytest.approx(1.0, abs=1e-12)
    assert S[0, 2] < 0.2


def _partition(groups):
    return sorted(tuple(sorted(gr)) for gr in groups)


def test_clustering_matches_library_average_linkage():
    g = np.random.default_rng(4)
    for h in (5, 8, 12):
        A = g.random((h, h))
        S = (A + A.T) / 2
        np.fill_diagonal(S, 1.0)
        Z = linkage(squareform(1.0 - S, checks=False), method="average")
        for K in range(1, h + 1):
            labels = fcluster(Z, K, criterion="maxclust")
            ref = [[i for i in range(h) if labels[i] == c] for c in sorted(set(labels))]
            if len(ref) != K:            # maxclust can stop early on equal heights
                continue
            assert _partition(oc.cluster_heads(S, K)) == _partition(ref), (h, K)


def test_clustering_extremes_and_blocks():
    S = np.full((6, 6), 0.1)
    for blk in ([0, 3], [1, 4, 5], [2]):
        for i in blk:
            for j in blk:
                S[i, j] = 0.9
    np.fill_diagonal(S, 1.0)
    assert oc.cluster_heads(S, 3) == [[0, 3], [1, 4, 5], [2]]
    assert oc.cluster_heads(S, 6) == [[i] for i in range(6)]
    assert oc.cluster_heads(S, 1) == [list(range(6))]
    assert oc.group_of_head([[0, 3], [1, 4, 5], [2]], 6) == [0, 1, 2, 0, 1, 1]


def test_energy_partitions_and_equals_singular_values():
    g = np.random.default_rng(5)
    W = g.standard_normal((30, 6 * 4))
    groups = [[0, 5], [1, 2, 3], [4]]
    Wg = oc.group_matrices(W, groups, 4)
    assert sum(oc.energy(Wi) for Wi in Wg) == pytest.approx(oc.energy(W), rel=1e-13)
    for Wi in Wg:
        assert oc.energy(Wi) == pytest.approx(np.sum(np.linalg.svd(Wi, compute_uv=False) ** 2), rel=1e-12)
    assert np.array_equal(Wg[0], np.concatenate([W[:, 0:4], W[:, 20:24]], axis=1))


def test_init_ranks_by_energy_hand_cases():
    # group energies 1 : 1 : 2 with r = 8 give 2, 2, 4
    W = np.zeros((4, 12))
    W[0, 0], W[1, 4], W[2, 8], W[3, 9] = 1.0, 1.0, 1.0, 1.0
    Wg = oc.group_matrices(W, [[0], [1], [2]], 4)
    assert oc.init_ranks_by_energy(Wg, W, 8) == [2, 2, 4]
    # 1 : 3 with r = 2: r E_i / E = 0.5 and 1.5 round half up to 1 and 2
    W2 = np.zeros((4, 8))
    W2[0, 0] = 1.0
    W2[1, 4] = np.sqrt(3.0)
    assert oc.init_ranks_by_energy(oc.group_matrices(W2, [[0], [1]], 4), W2, 2) == [1, 2]
    # a group with negligible energy still keeps rank 1; no rank exceeds min(m, h_i d_h)
    W3 = np.zeros((3, 8))
    W3[:, 4:] = 1.0
    W3[0, 0] = 1e-9
    assert oc.init_ranks_by_energy(oc.group_matrices(W3, [[0], [1]], 4), W3, 10) == [1, 3]


def test_greedy_adjust_hand_worked():
    # heads (1, 3), h = 4, r = 8: the budget needs r0 + 3 r1 <= 32 and r0 + r1 <= 8.
    # costs sigma^2 / alpha: group 0 drop = 4.5^2 * 4 = 81; group 1 drops
    # 1^2 * 4/3, 2^2 * 4/3, 3^2 * 4/3, 4^2 * 4/3 (all below 81): four steps on group 1.
    sig0 = np.array([5.0, 4.5])
    sig1 = np.arange(10, 0, -1, dtype=float)
    out = oc.greedy_adjust([2, 10], [sig0, sig1], [1, 3], 8)
    assert out == [2, 6]
    assert oc.budget_holds(out, [1, 3], 8)
    # from [2, 12] the last step lowers group 1 from rank 7 (cost 6^2 * 4/3 = 48
    # against 81); an unnormalised rule would compare 36 with 4.5^2 = 20.25 and
    # lower group 0 instead, ending at [1, 7]
    out2 = oc.greedy_adjust([2, 12], [sig0, np.arange(12, 0, -1, dtype=float)], [1, 3], 8)
    assert out2 == [2, 6]


def test_greedy_adjust_paper_budget_alone():
    # A case where only the paper's inequality binds (sum r_i = 8 = r from the
    # start, so the extra sum r_i <= r condition never acts): heads (2, 6),
    # h = 8, r = 8, so sum r_i h_i <= 4 r = 32 is required; start [2, 6] gives 40.
    # Costs sigma^2 / alpha: group 0 at rank 2: 2^2 * 8/2 = 16; group 1 at rank
    # 6: 2^2 * 8/6 = 5.33, then at rank 5: 2.5^2 * 8/6 = 8.33 -- group 1 twice,
    # ending at [2, 4] (4 + 24 = 28 <= 32).  An unnormalised rule ties 4 = 4 at
    # the first step, lowers group 0 and ends at [1, 5].
    sig0 = np.array([3.0, 2.0])
    sig1 = np.array([6.0, 5.0, 4.0, 3.0, 2.5, 2.0])
    assert not oc.budget_holds([2, 6], [2, 6], 8)
    assert oc.greedy_adjust([2, 6], [sig0, sig1], [2, 6], 8) == [2, 4]
    assert oc.greedy_cost(sig0, 2, 2, 8) == pytest.approx(16.0)
    assert oc.greedy_cost(sig1, 6, 6, 8) == pytest.approx(16.0 / 3.0)


def test_linkage_distance_is_the_pair_mean():
    D = np.array([[0.0, 0.2, 0.4, 0.9],
                  [0.2, 0.0, 0.6, 0.5],
                  [0.4, 0.6, 0.0, 0.3],
                  [0.9, 0.5, 0.3, 0.0]])
    assert oc.linkage_distance(D, [0, 1], [2]) == pytest.approx(0.5)
    assert oc.linkage_distance(D, [0, 1], [2, 3]) == pytest.approx((0.4 + 0.9 + 0.6 + 0.5) / 4)
    assert oc.linkage_distance(D, [3], [0]) == pytest.approx(0.9)


def test_group_decompose_eckart_young_and_balance():
    g = np.random.default_rng(6)
    Wi = g.standard_normal((20, 12))
    lam = np.sort(np.linalg.eigvalsh(Wi.T @ Wi))[::-1]          # sigma^2 by another routine
    for r in (1, 3, 7, 12):
        L, R = oc.group_decompose(Wi, r)
        assert L.shape == (20, r) and R.shape == (r, 12)
        assert np.sum((Wi - L @ R) ** 2) == pytest.approx(max(0.0, lam[r:].sum()), abs=1e-9)
        # balanced factors: L^T L = R R^T = diag(sigma_1..sigma_r)
        assert np.allclose(L.T @ L, np.diag(np.sqrt(lam[:r])), atol=1e-9)
        assert np.allclose(R @ R.T, np.diag(np.sqrt(lam[:r])), atol=1e-9)


def _planted(seed, group_heads, m=48, d=4, k=3, N=300):
    g = np.random.default_rng(seed)
    h = sum(len(x) for x in group_heads)
    W = np.zeros((m, h * d))
    for heads in group_heads:
        B = g.standard_normal((m, k))
        for hh in heads:
            W[:, hh * d:(hh + 1) * d] = B @ g.standard_normal((k, d))
    X = g.standard_normal((N, m))
    return W, X @ W


def test_compress_planted_groups_and_budget():
    groups = [[0, 4, 5], [1, 3], [2, 6, 7]]
    W, acts = _planted(7, groups)
    S = oc.head_similarity(acts, 8, 4)
    assert oc.cluster_heads(S, 3) == [[0, 4, 5], [1, 3], [2, 6, 7]]
    m, n, h, r = 48, 32, 8, 12
    res = oc.compress(W, S, r, [2, 3, 4, 5], 4)
    objs = [d["objective"] for d in res["all"]]
    assert res["best"]["objective"] == min(objs)
    for d in res["all"]:
        assert oc.budget_holds(d["ranks"], d["heads"], r)
        assert sum(d["ranks"]) <= r
        # the final count (greedy-adjusted) never exceeds the fixed four-head count
        assert params.final_params(m, n, d["ranks"], d["heads"]) <= params.fixed_group_params(m, r, n, h)
        assert d["objective"] == pytest.approx(d["error"] + (r - sum(d["ranks"])), rel=1e-12)
    # at K = 3 the planted rank-3 groups come back whole, every rank covers
    # its group's rank 3, so the error vanishes and the full budget is used:
    # objective 0, which no candidate beats (ties go to the smaller K)
    k3 = [d for d in res["all"] if d["K"] == 3][0]
    assert k3["groups"] == groups and min(k3["ranks"]) >= 3 and sum(k3["ranks"]) == r
    assert k3["error"] == pytest.approx(0.0, abs=1e-20 * oc.energy(W))
    assert res["best"]["K"] == 3
