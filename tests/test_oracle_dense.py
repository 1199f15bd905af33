"""Pins of the oracle's uncompressed decode (the baseline of the comparison):
against torch's scaled_dot_product_attention, its page layout, and the
compressed oracle in the full-rank case."""

import numpy as np
import pytest
import torch

from oracle import attention, dense, layout
from oracle.bookkeeping import make_book


def _pages(lens, g):
    pages = [-(-T // 64) for T in lens]
    table = np.zeros((len(lens), max(pages + [1])), dtype=np.int32)
    perm = g.permutation(sum(pages))
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    return table, sum(pages)


@pytest.mark.parametrize("Hq, Hkv, d, lens", [(4, 4, 8, [70, 1, 0]), (8, 2, 16, [130, 64]),
                                              (6, 3, 4, [200])])
def test_dense_equals_sdpa(Hq, Hkv, d, lens):
    g = np.random.default_rng(5)
    table, npages = _pages(lens, g)
    pool = dense.new_pool(npages, Hkv, d)
    Ks, Vs = [], []
    for b, T in enumerate(lens):
        K = g.standard_normal((T, Hkv, d))
        V = g.standard_normal((T, Hkv, d))
        dense.pack(pool, table, b, 0, K, V)
        Ks.append(K)
        Vs.append(V)
    q = g.standard_normal((len(lens), Hq, d))
    got = dense.decode(q, pool, table, lens, Hkv)
    for b, T in enumerate(lens):
        if T == 0:
            assert np.all(got[b] == 0)
            continue
        Kt = torch.from_numpy(Ks[b]).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0).contiguous()
        Vt = torch.from_numpy(Vs[b]).permute(1, 0, 2).repeat_interleave(Hq // Hkv, 0).contiguous()
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q[b]).view(Hq, 1, d), Kt, Vt).view(Hq, d).numpy()
        np.testing.assert_allclose(got[b], ref, rtol=1e-10, atol=1e-12)


def test_dense_layout_is_a_bijection_with_contiguous_heads():
    Hkv, d = 3, 8
    n = dense.page_elems(Hkv, d)
    s = np.arange(64)[:, None, None]
    kv = np.arange(Hkv)[None, :, None]
    dd = np.arange(d)[None, None, :]
    used = np.zeros(n, dtype=int)
    np.add.at(used, dense.key_offset(s, kv, dd, Hkv, d).ravel(), 1)
    np.add.at(used, dense.value_offset(s, kv, dd, Hkv, d).ravel(), 1)
    assert np.all(used == 1)
    # one head's keys of a page: 64 * d contiguous elements
    offs = dense.key_offset(s, 1, dd, Hkv, d).ravel()
    assert np.array_equal(np.sort(offs), np.arange(64 * d, 2 * 64 * d))


def test_dense_equals_compressed_oracle_at_full_rank():
    # exact factorisations: decode over latents and decode over K = x W_k,
    # V = x W_v must agree (two independent code paths of the oracle)
    g = np.random.default_rng(9)
    Hq, Hkv, d, m, T = 8, 4, 4, 24, 90
    gmap = [0, 1, 1, 0]
    bk = make_book(m, Hq, Hkv, d, gmap, [8, 8], Hkv * d)
    W_k = g.standard_normal((m, Hkv * d))
    W_v = g.standard_normal((m, Hkv * d))
    R_blocks, L_blocks = [], []
    for grp in range(2):
        cols = np.concatenate([np.arange(kv * d, (kv + 1) * d) for kv in bk.members[grp]])
        Q_, r_ = np.linalg.qr(g.standard_normal((len(cols), len(cols))))
        R_g = Q_ * np.sign(np.diag(r_))[None, :]
        L_blocks.append(W_k[:, cols] @ R_g.T)
        R_blocks.append(R_g)
    Q_, r_ = np.linalg.qr(g.standard_normal((Hkv * d, Hkv * d)))
    R_v = Q_ * np.sign(np.diag(r_))[None, :]
    x = g.standard_normal((T, m))
    table = np.array([[1, 0]], dtype=np.int32)
    lat = layout.new_pool(2, bk.key_rank_total, Hkv * d)
    layout.pack(lat, table, 0, 0, x @ np.concatenate(L_blocks, axis=1), x @ (W_v @ R_v.T))
    den = dense.new_pool(2, Hkv, d)
    dense.pack(den, table, 0, 0, (x @ W_k).reshape(T, Hkv, d), (x @ W_v).reshape(T, Hkv, d))
    q = g.standard_normal((1, Hq, d))
    a = attention.decode(q, lat, table, [T], R_blocks, R_v, bk, chunk=None)
    b = dense.decode(q, den, table, [T], Hkv)
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
