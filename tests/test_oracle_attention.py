"""Pins of the oracle's decode attention.

The anchor is the full-rank special case of the latent caching (Sec. III-A):
when every factorisation is exact (W_g = L_g R_g with square orthogonal R_g,
W_v = L_v R_v with orthogonal R_v), decode over the latents must equal plain
attention with K = x W_k and V = x W_v, computed here by the library routine
torch.nn.functional.scaled_dot_product_attention in fp64.  Closed forms,
invariances, a scalar brute force and planted mistakes complete the set.
"""

import copy
import math

import numpy as np
import pytest
import torch

from oracle import attention, layout
from oracle.bookkeeping import make_book


def _orth(g, n):
    q, r = np.linalg.qr(g.standard_normal((n, n)))
    return q * np.sign(np.diag(r))[None, :]


def _full_rank_case(seed, H_q, H_kv, d, gmap, m, lens):
    g = np.random.default_rng(seed)
    G = max(gmap) + 1
    sizes = [list(gmap).count(i) for i in range(G)]
    ranks = [s * d for s in sizes]
    n = H_kv * d
    bk = make_book(m, H_q, H_kv, d, gmap, ranks, n)
    W_k = g.standard_normal((m, n))
    W_v = g.standard_normal((m, n))
    L_blocks, R_blocks = [], []
    for grp in range(G):
        cols = np.concatenate([np.arange(kv * d, (kv + 1) * d) for kv in bk.members[grp]])
        W_g = W_k[:, cols]
        R_g = _orth(g, len(cols))
        L_blocks.append(W_g @ R_g.T)
        R_blocks.append(R_g)
    L_keys = np.concatenate(L_blocks, axis=1)
    R_v = _orth(g, n)
    L_v = W_v @ R_v.T
    B = len(lens)
    q = g.standard_normal((B, H_q, d))
    xs = [g.standard_normal((T, m)) for T in lens]
    pages = [-(-T // 64) for T in lens]
    table = np.zeros((B, max(pages) if pages else 1), dtype=np.int32)
    perm = g.permutation(sum(pages))
    pos = 0
    for b, npg in enumerate(pages):
        table[b, :npg] = perm[pos:pos + npg]
        pos += npg
    pool = layout.new_pool(sum(pages), bk.key_rank_total, n)
    for b, x in enumerate(xs):
        layout.pack(pool, table, b, 0, x @ L_keys, x @ L_v)
    return dict(bk=bk, W_k=W_k, W_v=W_v, R_blocks=R_blocks, R_v=R_v, q=q, xs=xs,
                table=table, pool=pool, lens=lens)


def _reference_sdpa(c):
    bk = c["bk"]
    H_q, H_kv, d = bk.num_q_heads, bk.num_kv_heads, bk.head_dim
    out = np.zeros(c["q"].shape)
    for b, x in enumerate(c["xs"]):
        T = x.shape[0]
        if T == 0:
            continue
        K = torch.from_numpy(x @ c["W_k"]).view(T, H_kv, d).permute(1, 0, 2)
        V = torch.from_numpy(x @ c["W_v"]).view(T, H_kv, d).permute(1, 0, 2)
        K = K.repeat_interleave(H_q // H_kv, dim=0).contiguous()
        V = V.repeat_interleave(H_q // H_kv, dim=0).contiguous()
        qq = torch.from_numpy(c["q"][b]).view(H_q, 1, d)
        o = torch.nn.functional.scaled_dot_product_attention(qq, K, V)
        out[b] = o.view(H_q, d).numpy()
    return out


def _oracle(c, bk=None):
    return attention.decode(c["q"], c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                            bk or c["bk"], chunk=None)


CASES = [
    # (H_q, H_kv, d, group map, m, lengths)
    (4, 4, 4, [1, 0, 1, 1], 24, [37]),                 # MHA, singleton + triple
    (8, 4, 4, [0, 1, 1, 0], 20, [70, 5]),              # GQA, two per KV head
    (12, 3, 2, [0, 0, 0], 8, [129, 64, 1]),            # GQA, one group holds all
    (6, 6, 3, [2, 0, 1, 2, 0, 2], 30, [90]),           # MHA, three uneven groups
]


@pytest.mark.parametrize("case", CASES)
def test_full_rank_equals_uncompressed_attention(case):
    c = _full_rank_case(1234, *case)
    np.testing.assert_allclose(_oracle(c), _reference_sdpa(c), rtol=1e-10, atol=1e-11)


def test_planted_mistakes_are_caught():
    # Each mutation of the oracle's bookkeeping must break the full-rank pin.
    c = _full_rank_case(99, 8, 4, 4, [0, 1, 1, 0], 20, [70])
    ref = _reference_sdpa(c)
    np.testing.assert_allclose(_oracle(c), ref, rtol=1e-10, atol=1e-11)
    mutants = []
    bk = copy.deepcopy(c["bk"]);   bk.pos_in_group = [1 - p for p in bk.pos_in_group]
    mutants.append(bk)                                          # reversed head order in groups
    bk = copy.deepcopy(c["bk"]);   bk.kv_of_q = [h % 4 for h in range(8)]
    mutants.append(bk)                                          # interleaved GQA map
    bk = copy.deepcopy(c["bk"]);   bk.koff = list(reversed(bk.koff))
    mutants.append(bk)                                          # wrong group latent columns
    for bk in mutants:
        assert not np.allclose(_oracle(c, bk), ref, rtol=1e-6, atol=1e-6)


def test_planted_scale_and_transpose_mistakes_are_caught(monkeypatch):
    c = _full_rank_case(5, 4, 4, 4, [1, 0, 1, 1], 24, [37])
    ref = _reference_sdpa(c)

    def attend_no_scale(q_h, K, V):
        s = K @ q_h
        p = np.exp(s - s.max())
        return (p / p.sum()) @ V
    monkeypatch.setattr(attention, "attend", attend_no_scale)
    assert not np.allclose(_oracle(c), ref, rtol=1e-6, atol=1e-6)
    monkeypatch.undo()

    orig = attention.key_up

    def key_up_transposed_rows(R_keys, book, h):
        R = orig(R_keys, book, h)
        return R[::-1]                                          # rows in the wrong order
    monkeypatch.setattr(attention, "key_up", key_up_transposed_rows)
    assert not np.allclose(_oracle(c), ref, rtol=1e-6, atol=1e-6)


def _random_case(seed, H_q=4, H_kv=2, d=3, gmap=(0, 1), ranks=(2, 3), rv=5, lens=(7,)):
    g = np.random.default_rng(seed)
    bk = make_book(16, H_q, H_kv, d, list(gmap), list(ranks), rv)
    R_blocks = [g.standard_normal((r, s * d)) for r, s in zip(ranks, bk.heads_per_group)]
    R_v = g.standard_normal((rv, H_kv * d))
    q = g.standard_normal((len(lens), H_q, d))
    Zs = [(g.standard_normal((T, sum(ranks))), g.standard_normal((T, rv))) for T in lens]
    table = np.arange(sum(-(-T // 64) for T in lens), dtype=np.int32)
    tbl = np.zeros((len(lens), max(1, max(-(-T // 64) for T in lens))), dtype=np.int32)
    pos = 0
    for b, T in enumerate(lens):
        npg = -(-T // 64)
        tbl[b, :npg] = table[pos:pos + npg]
        pos += npg
    pool = layout.new_pool(max(1, pos), sum(ranks), rv)
    for b, (Zk, Zv) in enumerate(Zs):
        layout.pack(pool, tbl, b, 0, Zk, Zv)
    return bk, R_blocks, R_v, q, Zs, tbl, pool, list(lens)


def test_brute_force_scalar_loops():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(3, lens=(9, 4))
    got = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk, chunk=None)
    d = bk.head_dim
    for b, (Zk, Zv) in enumerate(Zs):
        T = lens[b]
        for h in range(bk.num_q_heads):
            kv = h // (bk.num_q_heads // bk.num_kv_heads)
            grp = bk.group_of_kv[kv]
            j = sorted(i for i in range(bk.num_kv_heads) if bk.group_of_kv[i] == grp).index(kv)
            col0 = sum(bk.ranks[:grp])
            s = []
            for t in range(T):
                acc = 0.0
                for c in range(d):
                    kval = 0.0
                    for r in range(bk.ranks[grp]):
                        kval += Zk[t, col0 + r] * R_blocks[grp][r, j * d + c]
                    acc += kval * q[b, h, c]
                s.append(acc / math.sqrt(d))
            mx = max(s)
            e = [math.exp(v - mx) for v in s]
            tot = sum(e)
            for c in range(d):
                o = 0.0
                for t in range(T):
                    vval = 0.0
                    for r in range(bk.value_rank):
                        vval += Zv[t, r] * R_v[r, kv * d + c]
                    o += e[t] / tot * vval
                assert abs(o - got[b, h, c]) < 1e-12 * (1 + abs(o))


def test_single_token_closed_form():
    # T = 1: the softmax weight is 1, so o_h = z_v R_v[:, kv block] for any q.
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(4, lens=(1,))
    got = attention.decode(q * 1e3, pool, tbl, lens, R_blocks, R_v, bk)
    for h in range(bk.num_q_heads):
        kv = h // 2
        np.testing.assert_allclose(got[0, h], Zs[0][1][0] @ R_v[:, kv * 3:(kv + 1) * 3], rtol=1e-13)


def test_zero_query_closed_form():
    # q = 0: all scores equal, so o_h is the mean value row.
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(5, lens=(130,))
    got = attention.decode(np.zeros_like(q), pool, tbl, lens, R_blocks, R_v, bk)
    for h in range(bk.num_q_heads):
        kv = h // 2
        np.testing.assert_allclose(got[0, h], Zs[0][1].mean(0) @ R_v[:, kv * 3:(kv + 1) * 3], rtol=1e-12)


def test_dominant_token_limit():
    # Scale q so one token's score dominates: o_h tends to that token's value.
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(6, lens=(50,))
    Zk, Zv = Zs[0]
    h = 0
    K, V = attention.rebuild(Zk, Zv, R_blocks, R_v, bk, h)
    qh = K[17] / np.linalg.norm(K[17])
    q2 = np.zeros_like(q)
    q2[0, h] = qh * 1e4
    got = attention.decode(q2, pool, tbl, lens, R_blocks, R_v, bk)
    t_star = int(np.argmax(K @ qh))
    np.testing.assert_allclose(got[0, h], V[t_star], rtol=1e-9, atol=1e-9)


def test_token_permutation_invariance():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(7, lens=(100,))
    base = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk)
    perm = np.random.default_rng(1).permutation(100)
    pool2 = layout.new_pool(pool.shape[0], bk.key_rank_total, bk.value_rank)
    layout.pack(pool2, tbl, 0, 0, Zs[0][0][perm], Zs[0][1][perm])
    got = attention.decode(q, pool2, tbl, lens, R_blocks, R_v, bk)
    np.testing.assert_allclose(got, base, rtol=1e-12, atol=1e-14)


def test_group_relabel_invariance():
    # Renumbering the groups (and moving their latent columns and factor
    # blocks with them) leaves the output unchanged.
    gmap, ranks = [2, 0, 1, 0, 2, 2], [3, 2, 4]
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(
        8, H_q=6, H_kv=6, d=2, gmap=gmap, ranks=ranks, rv=4, lens=(33,))
    base = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk)
    relabel = [1, 2, 0]                       # old group -> new group
    inv = [relabel.index(i) for i in range(3)]
    gmap2 = [relabel[g_] for g_ in gmap]
    ranks2 = [ranks[inv[i]] for i in range(3)]
    bk2 = make_book(16, 6, 6, 2, gmap2, ranks2, 4)
    R2 = [R_blocks[inv[i]] for i in range(3)]
    Zk = Zs[0][0]
    cols = np.concatenate([np.arange(bk.koff[inv[i]], bk.koff[inv[i]] + ranks[inv[i]]) for i in range(3)])
    pool2 = layout.new_pool(pool.shape[0], sum(ranks), 4)
    layout.pack(pool2, tbl, 0, 0, Zk[:, cols], Zs[0][1])
    got = attention.decode(q, pool2, tbl, lens, R2, R_v, bk2)
    np.testing.assert_allclose(got, base, rtol=1e-12, atol=1e-14)


def test_chunked_equals_whole_and_empty_sequence():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(9, lens=(300, 0, 65))
    whole = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk, chunk=None)
    chunked = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk, chunk=64)
    np.testing.assert_allclose(chunked, whole, rtol=1e-12, atol=1e-14)
    assert np.all(whole[1] == 0)
    part = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk, pairs=[(2, 1)])
    np.testing.assert_array_equal(part[2, 1], whole[2, 1])
    assert np.isnan(part[0]).all()


def test_flat_and_blocked_factor_forms_agree():
    bk, R_blocks, R_v, q, Zs, tbl, pool, lens = _random_case(10, lens=(40,))
    flat = np.concatenate([b.reshape(-1) for b in R_blocks])
    a = attention.decode(q, pool, tbl, lens, R_blocks, R_v, bk)
    b = attention.decode(q, pool, tbl, lens, flat, R_v, bk)
    np.testing.assert_array_equal(a, b)


# ---------------------------------------------------- several queries a sequence
def _reference_sdpa_causal_tail(c, qm):
    """Causal attention over the whole sequence with the last Q query rows
    replaced by qm[b] (Q x H_q x d); returns those Q rows."""
    bk = c["bk"]
    H_q, H_kv, d = bk.num_q_heads, bk.num_kv_heads, bk.head_dim
    Q = qm.shape[1]
    out = np.zeros(qm.shape)
    for b, x in enumerate(c["xs"]):
        T = x.shape[0]
        K = torch.from_numpy(x @ c["W_k"]).view(T, H_kv, d).permute(1, 0, 2)
        V = torch.from_numpy(x @ c["W_v"]).view(T, H_kv, d).permute(1, 0, 2)
        K = K.repeat_interleave(H_q // H_kv, dim=0).contiguous()
        V = V.repeat_interleave(H_q // H_kv, dim=0).contiguous()
        qq = torch.zeros(H_q, T, d, dtype=torch.float64)
        qq[:, T - Q:, :] = torch.from_numpy(qm[b]).permute(1, 0, 2)
        o = torch.nn.functional.scaled_dot_product_attention(qq, K, V, is_causal=True)
        out[b] = o[:, T - Q:, :].permute(1, 0, 2).numpy()
    return out


@pytest.mark.parametrize("case, Q", [(CASES[0], 3), (CASES[1], 5), (CASES[3], 8)])
def test_multi_query_equals_causal_attention_tail(case, Q):
    c = _full_rank_case(4321, *case)
    bk = c["bk"]
    g = np.random.default_rng(8)
    qm = g.standard_normal((len(c["lens"]), Q, bk.num_q_heads, bk.head_dim))
    got = attention.decode_multi(qm, c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                                 bk, chunk=None)
    np.testing.assert_allclose(got, _reference_sdpa_causal_tail(c, qm), rtol=1e-10, atol=1e-11)


def test_multi_query_special_cases():
    c = _full_rank_case(77, *CASES[1])
    bk = c["bk"]
    g = np.random.default_rng(2)
    B, Q = len(c["lens"]), 4
    qm = g.standard_normal((B, Q, bk.num_q_heads, bk.head_dim))
    got = attention.decode_multi(qm, c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                                 bk, chunk=None)
    # the last query sees the whole sequence: the single-query decode
    last = attention.decode(qm[:, -1], c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                            bk, chunk=None)
    np.testing.assert_allclose(got[:, -1], last, rtol=1e-12, atol=1e-13)
    # sequence 1 holds 5 tokens: query 0 of 4 sees 2 of them, and with Q > T
    # the first queries see nothing
    assert attention.visible_tokens(5, 4, 0) == 2 and attention.visible_tokens(5, 8, 2) == 0
    qm8 = g.standard_normal((B, 8, bk.num_q_heads, bk.head_dim))
    got8 = attention.decode_multi(qm8, c["pool"], c["table"], c["lens"], c["R_blocks"], c["R_v"],
                                  bk, chunk=None)
    assert np.all(got8[1, :3] == 0) and np.all(np.abs(got8[1, 3:]).sum(axis=-1) > 0)
    # a query that sees one token returns that token's value (T = 5, Q = 8, i = 3)
    V = c["xs"][1] @ c["W_v"]
    for h in range(bk.num_q_heads):
        kv = h // (bk.num_q_heads // bk.num_kv_heads)
        np.testing.assert_allclose(got8[1, 3, h], V[0, kv * bk.head_dim:(kv + 1) * bk.head_dim],
                                   rtol=1e-10, atol=1e-12)
