"""Pins of the paged latent layout (a stated reading; the paper fixes none)."""

import numpy as np
import pytest

from oracle import layout


@pytest.mark.parametrize("RK, rv", [(1, 1), (7, 3), (8, 8), (43, 17), (128, 128), (1228, 1536)])
def test_offsets_are_a_bijection_onto_the_page(RK, rv):
    RKp = layout.key_width_padded(RK)
    rvp = layout.value_width_padded(rv)
    assert RKp % 32 == 0 and RK <= RKp < RK + 32
    assert rvp % 16 == 0 and rv <= rvp < rv + 16
    n = layout.page_elems(RK, rv)
    assert n == 64 * (RKp + rvp)
    used = np.zeros(n, dtype=np.int64)
    s = np.arange(64)[:, None]
    used_k = layout.key_offset(s, np.arange(RK)[None, :], RK).ravel()
    used_v = layout.value_offset(s, np.arange(rv)[None, :], RK).ravel()
    np.add.at(used, used_k, 1)
    np.add.at(used, used_v, 1)
    # every latent element has its own slot; the only unused slots are the
    # key padding columns RK..RKp-1 and value padding columns rv..rvp-1
    assert used.max() == 1
    pad = np.flatnonzero(used == 0)
    expect_pad = np.concatenate([layout.key_offset(s, np.arange(RK, RKp)[None, :], RK).ravel(),
                                 layout.value_offset(s, np.arange(rv, rvp)[None, :], RK).ravel()])
    assert np.array_equal(np.sort(pad), np.sort(expect_pad))


def test_hand_offsets():
    # R_K = 40 -> two chunks of 32 (64 padded columns); r_v = 3 -> one tile of 16
    assert layout.key_width_padded(40) == 64
    assert layout.value_width_padded(3) == 16
    assert layout.page_elems(40, 3) == 64 * 64 + 64 * 16
    assert layout.key_offset(0, 0, 40) == 0
    assert layout.key_offset(0, 31, 40) == 31
    assert layout.key_offset(1, 0, 40) == 32           # next slot, same chunk
    assert layout.key_offset(2, 33, 40) == 2048 + 2 * 32 + 1   # second chunk
    assert layout.value_offset(0, 0, 40) == 4096
    assert layout.value_offset(5, 2, 40) == 4096 + 2 * 32 + 5          # first half of tile 0
    assert layout.value_offset(33, 2, 40) == 4096 + 512 + 2 * 32 + 1   # second half
    assert layout.value_offset(33, 17, 40) == 4096 + 1024 + 512 + 32 + 1   # tile 1


def test_mfma_tile_is_contiguous():
    # 16 consecutive slots x one 32-column chunk occupy 1 KB of bf16 in one run
    offs = layout.key_offset(np.arange(16, 32)[:, None], np.arange(64, 96)[None, :], 100)
    assert np.array_equal(np.sort(offs.ravel()), np.arange(offs.min(), offs.min() + 512))


def test_value_mfma_tile_is_contiguous():
    # 16 value columns of one tile x 32 slots of one half: 1 KB of bf16 in one run
    for j0, s0 in ((0, 0), (16, 32), (48, 0)):
        offs = layout.value_offset(np.arange(s0, s0 + 32)[None, :], np.arange(j0, j0 + 16)[:, None], 100)
        assert np.array_equal(np.sort(offs.ravel()), np.arange(offs.min(), offs.min() + 512))


def test_pack_unpack_through_permuted_pages():
    g = np.random.default_rng(0)
    RK, rv, lens = 13, 9, [1, 64, 65, 200]
    pages = [-(-t // 64) for t in lens]
    phys = g.permutation(sum(pages))
    table = np.zeros((len(lens), max(pages)), dtype=np.int32)
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = phys[pos:pos + n]
        pos += n
    pool = layout.new_pool(sum(pages), RK, rv)
    data = []
    for b, T in enumerate(lens):
        Zk = g.standard_normal((T, RK))
        Zv = g.standard_normal((T, rv))
        # write in two uneven pieces to cross page boundaries mid-call
        cut = T // 3
        layout.pack(pool, table, b, 0, Zk[:cut], Zv[:cut])
        layout.pack(pool, table, b, cut, Zk[cut:], Zv[cut:])
        data.append((Zk, Zv))
    for b, T in enumerate(lens):
        Zk, Zv = layout.unpack(pool, table, b, T, RK, rv)
        assert np.array_equal(Zk, data[b][0]) and np.array_equal(Zv, data[b][1])
        # element-by-element against the offset functions
        for t in range(0, T, 17):
            page, s = table[b, t // 64], t % 64
            for k in range(RK):
                assert pool[page, layout.key_offset(s, k, RK)] == data[b][0][t, k]
            for j in range(rv):
                assert pool[page, layout.value_offset(s, j, RK)] == data[b][1][t, j]
    # untouched slots (padding columns, slots past each length) stay zero
    written = np.zeros_like(pool, dtype=bool)
    for b, T in enumerate(lens):
        for t in range(T):
            page, s = table[b, t // 64], t % 64
            written[page, layout.key_offset(s, np.arange(RK), RK)] = True
            written[page, layout.value_offset(s, np.arange(rv), RK)] = True
    assert np.all(pool[~written] == 0)
