"""Pins of the head/group bookkeeping (Sec. III-C column-wise head groups)."""

import itertools

import pytest

from oracle.bookkeeping import PartitionError, group_members, make_book


def test_tiny_layer_by_hand():
    # heads {0,2,4,6} -> group 0 (rank 48), {1,3,5,7} -> group 1 (rank 80)
    bk = make_book(512, 8, 8, 64, [0, 1, 0, 1, 0, 1, 0, 1], [48, 80], 128)
    assert bk.members == [[0, 2, 4, 6], [1, 3, 5, 7]]
    assert bk.heads_per_group == [4, 4]
    assert bk.pos_in_group == [0, 0, 1, 1, 2, 2, 3, 3]
    assert bk.koff == [0, 48]
    assert bk.roff == [0, 48 * 256, 48 * 256 + 80 * 256]
    assert bk.kv_of_q == list(range(8))
    assert bk.qoff == [0, 48, 128, 176, 256, 304, 384, 432, 512]
    assert [float(a) for a in bk.alpha] == [0.5, 0.5]


def test_grouped_query_map():
    # 8 query heads over 2 KV heads: heads 0-3 read KV 0, heads 4-7 read KV 1
    bk = make_book(64, 8, 2, 16, [1, 0], [10, 7], 20)
    assert bk.kv_of_q == [0, 0, 0, 0, 1, 1, 1, 1]
    assert bk.group_of_q == [1, 1, 1, 1, 0, 0, 0, 0]
    assert bk.qoff == [0, 7, 14, 21, 28, 38, 48, 58, 68]
    assert bk.pos_in_group == [0, 0]


def test_every_surjective_map_is_a_partition():
    # Exhaustive over all maps of 5 heads onto up to 4 groups: a map is
    # accepted exactly when it is onto, and then every head sits in exactly
    # one group at a position that lists the group's heads in ascending order.
    H = 5
    for G in range(1, 5):
        for gmap in itertools.product(range(G), repeat=H):
            onto = set(gmap) == set(range(G))
            if not onto:
                with pytest.raises(PartitionError):
                    group_members(gmap, G)
                continue
            mem = group_members(gmap, G)
            flat = sorted(h for m in mem for h in m)
            assert flat == list(range(H))
            assert sum(len(m) for m in mem) == H
            bk = make_book(64, H, H, 4, gmap, [1] * G, 4)
            for g, m in enumerate(mem):
                assert m == sorted(m)
                for j, kv in enumerate(m):
                    assert bk.pos_in_group[kv] == j and bk.group_of_kv[kv] == g


@pytest.mark.parametrize("kw", [
    dict(ranks=[0, 4]),                 # empty rank
    dict(ranks=[4 * 16 + 1, 4]),        # rank above h_g d_h
    dict(num_q=6),                      # query heads not a multiple of KV heads
    dict(gmap=[0, 0, 0, 0]),            # group 1 empty
    dict(gmap=[0, 1, 2, 0]),            # group id out of range
    dict(value_rank=0),
    dict(value_rank=65),                # above n
    dict(hidden=3),                     # rank above m
])
def test_rejections(kw):
    args = dict(hidden=64, num_q=4, gmap=[0, 1, 0, 1], ranks=[4, 4], value_rank=16)
    args.update(kw)
    with pytest.raises(PartitionError):
        make_book(args["hidden"], args["num_q"], 4, 16, args["gmap"], args["ranks"], args["value_rank"])
