"""GPU parity of the offline compression calls (Sec. III-A, III-C, III-D)
against the fp64 oracle: the Gram matrix (centred and plain, fp32 and bf16
samples, ragged tiles), the CKA head similarity, and the two pipelines
(Algorithm 1 for keys, the calibration refinement for values)."""

import numpy as np
import pytest
import torch

from oracle import calibrate as ocal
from oracle import compress as oc

import decisions

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _gram_bound(A64, center, rows):
    # fp32 rounding of the centring (means, differences) and of a sum of
    # `rows` products: |dG| <= gamma * sum_t (|a_ti| + |mu_i|)(|a_tj| + |mu_j|)
    mu = np.abs(A64.mean(axis=0)) if center else np.zeros(A64.shape[1])
    M = np.abs(A64) + mu[None, :]
    gamma = 2.0 * (rows + 8) * U32
    return gamma * (M.T @ M) + 1e-30


# (rows, cols, dtype, centre): ragged sample counts (not a multiple of the
# 32-sample step), column counts that leave partial 128-column tiles, one
# sample, the smallest width; 4000 columns take the 192-column tiles (the
# last one partial)
CASES = [(200, 72, "f32", True), (1000, 264, "f32", True), (1000, 264, "f32", False),
         (37, 8, "f32", True), (513, 392, "bf16", True), (1, 16, "f32", True),
         (2048, 256, "bf16", False), (100, 4000, "f32", True), (70, 4000, "bf16", False)]


@pytest.mark.parametrize("rows, cols, dtype, center", CASES)
def test_gram_matches_oracle(rows, cols, dtype, center):
    from paper_2607_24331_amd import gram
    g = np.random.default_rng(rows * 7 + cols)
    A = (g.standard_normal((rows, cols)) + g.standard_normal(cols)[None, :]).astype(np.float32)
    At = torch.from_numpy(A).cuda()
    if dtype == "bf16":
        At = At.to(torch.bfloat16)
        A = At.float().cpu().numpy()                        # the values the GPU sees
    print(f"[gram] rows {rows} cols {cols} {dtype} center {center}", flush=True)
    G = gram(At, center=center)
    torch.cuda.synchronize()
    got = G.double().cpu().numpy()
    A64 = A.astype(np.float64)
    ref = ocal.gram(oc.centered(A64) if center else A64)
    assert np.all(np.abs(got - ref) <= _gram_bound(A64, center, rows))
    assert np.array_equal(got, got.T)                       # mirrored tiles are exact copies


def test_gram_is_bitwise_reproducible():
    from paper_2607_24331_amd import gram
    A = torch.randn(777, 200, device="cuda")
    a = gram(A).clone()
    b = gram(A)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def _acts(seed, h, d, N, groups):
    # per-head activations X W_h with heads of one planted group sharing a subspace
    g = np.random.default_rng(seed)
    m = 64
    W = np.zeros((m, h * d))
    for grp in groups:
        B = g.standard_normal((m, 6))
        for hh in grp:
            W[:, hh * d:(hh + 1) * d] = B @ g.standard_normal((6, d)) + 0.3 * g.standard_normal((m, d))
    X = g.standard_normal((N, m))
    return W, (X @ W + 0.5).astype(np.float32)


def test_head_similarity_matches_oracle():
    from paper_2607_24331_amd.offline import key_similarity
    for h, d, N in [(8, 16, 300), (12, 64, 1000), (5, 8, 77)]:
        groups = [list(range(0, h, 3)), list(range(1, h, 3)), list(range(2, h, 3))]
        _, acts = _acts(h * d, h, d, N, groups)
        print(f"[sim] h {h} d {d} N {N}", flush=True)
        S = key_similarity(torch.from_numpy(acts).cuda(), h, d)
        torch.cuda.synchronize()
        ref = oc.head_similarity(acts.astype(np.float64), h, d)
        Sh = S.double().cpu().numpy()
        assert np.max(np.abs(Sh - ref)) <= 1e-4
        assert np.array_equal(Sh, Sh.T)                     # CKA is symmetric: exactly so here


def test_head_similarity_full_size_sampled():
    # 32 heads x 128 over 2048 samples: S in full, the Gram on sampled rows
    from paper_2607_24331_amd import gram, head_similarity
    h, d, N = 32, 128, 2048
    groups = [list(range(k, h, 4)) for k in range(4)]
    _, acts = _acts(99, h, d, N, groups)
    At = torch.from_numpy(acts).cuda()
    G = gram(At, center=True)
    S = head_similarity(G, h, d)
    torch.cuda.synchronize()
    ref = oc.head_similarity(acts.astype(np.float64), h, d)
    assert np.max(np.abs(S.double().cpu().numpy() - ref)) <= 1e-4
    A64 = oc.centered(acts.astype(np.float64))
    rows = np.random.default_rng(5).choice(h * d, 48, replace=False)
    ref_rows = A64[:, rows].T @ A64
    bound = _gram_bound(acts.astype(np.float64), True, N)[rows]
    assert np.all(np.abs(G.double().cpu().numpy()[rows] - ref_rows) <= bound)


def test_compress_keys_matches_oracle():
    from paper_2607_24331_amd import cluster_merges
    from paper_2607_24331_amd.offline import compress_keys, key_similarity
    h, d = 12, 8
    groups = [[0, 4, 7, 9], [1, 2, 10], [3, 5, 6, 8, 11]]
    W, acts = _acts(7, h, d, 600, groups)
    S = key_similarity(torch.from_numpy(acts).cuda(), h, d).double().cpu().numpy()
    r, cands = 40, [2, 3, 4, 6]
    got = compress_keys(W, S, r, cands, d)
    ref = oc.compress(W, S, r, cands, d)             # the same S: the same decisions
    # decisions: the library's merge path is the oracle's up to near-ties
    # (tests/decisions.py); where no near-tie alternative was taken the
    # groups, ranks and objectives are identical
    merges = cluster_merges(S)
    first_dev = decisions.check_merges(S, merges)
    for a, b in zip(got["all"], ref["all"]):
        K = a["K"]
        gid = decisions.cut(merges, h, K)
        assert a["groups"] == [[x for x in range(h) if gid[x] == k] for k in range(K)]
        Wg = oc.group_matrices(W, a["groups"], d)
        sig = [np.linalg.svd(Wi, compute_uv=False) for Wi in Wg]
        assert decisions.init_ranks_agree(a["init_ranks"], [oc.energy(Wi) for Wi in Wg], oc.energy(W),
                                          [min(Wi.shape) for Wi in Wg], r)
        reachable, exact = decisions.greedy_reachable(a["init_ranks"], sig, a["heads"], r, a["ranks"])
        assert reachable
        factors = [oc.group_decompose(Wi, ri) for Wi, ri in zip(Wg, a["ranks"])]
        assert a["objective"] == pytest.approx(oc.objective(Wg, factors, a["ranks"], r), rel=1e-9, abs=1e-9)
        for (La, Ra), (Lb, Rb) in zip(a["factors"], factors):
            assert np.allclose(La @ Ra, Lb @ Rb, atol=1e-9)
        if h - K <= first_dev and exact:
            assert a["groups"] == b["groups"] and a["ranks"] == b["ranks"]
            assert a["init_ranks"] == b["init_ranks"]
            assert a["objective"] == pytest.approx(b["objective"], rel=1e-9, abs=1e-9)
    objs = [a["objective"] for a in got["all"]]
    assert got["best"]["objective"] == min(objs)
    assert got["best"]["K"] == min(a["K"] for a in got["all"] if a["objective"] == min(objs))
    assert first_dev == h - 1 and got["best"]["K"] == ref["best"]["K"]   # continuous S: no near-ties
    assert oc.cluster_heads(S, 3) == groups


def test_refine_value_matches_oracle():
    from paper_2607_24331_amd.offline import refine_value
    g = np.random.default_rng(8)
    m, n, N, r = 64, 48, 700, 12
    W = g.standard_normal((m, n))
    X = (g.standard_normal((N, m)) * np.logspace(0, 1, m)[None, :]).astype(np.float32)
    got = refine_value(W, r, torch.from_numpy(X).cuda())
    ref = ocal.refine(X.astype(np.float64), W, r)
    # the GPU Gram is fp32: the refined product agrees to fp32-level relative error
    scale = np.max(np.abs(ref["L"] @ ref["R"]))
    assert np.max(np.abs(got["L"] @ got["R"] - ref["L"] @ ref["R"])) <= 1e-4 * scale
    assert got["eps"] <= got["eps_mid"] * (1 + 1e-6) <= got["eps_svd"] * (1 + 1e-6)
    assert got["eps"] == pytest.approx(ref["eps"], rel=1e-4)
