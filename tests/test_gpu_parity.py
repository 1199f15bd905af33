"""GPU parity of latent_append and decode against the CPU oracle.

Small cases compare every output row and span several page tiles, splits,
ragged tails, singleton groups, odd ranks, GQA and permuted pages; the
full-size workloads compare sampled rows the oracle computes one by one.
Tolerances: attention rows within 2e-2 relative (bf16 latents, fp32
accumulation), 1e-4 for fp32 latents; latent writes bit-exact on
exact-arithmetic inputs and otherwise within one bf16 ulp plus the fp32
accumulation bound.
"""

import numpy as np
import pytest
import torch

from oracle import append as oappend
from oracle import attention as oattn
from oracle import bf16 as obf16
from oracle import layout as olayout
from oracle.bookkeeping import book_for
from workloads import WORKLOAD_NAMES, make_workload
from workloads.configs import custom_workload
from workloads.inputs import bf16_bits_from_f32, make_inputs

from gpu_common import (TOL_REL_ROW, TOL_REL_ROW_F32, dev, gpu_pool_with_append, oracle_pool,
                        oracle_rows, plan_for, row_rel_err, run_decode, sample_pairs, append_slots)

pytestmark = pytest.mark.gpu


def _report(name, errs):
    print(f"[parity] {name}: max row rel err {max(errs):.3e} over {len(errs)} rows", flush=True)


def _groups(sizes, seed):
    g = np.random.default_rng(seed)
    perm = g.permutation(sum(sizes))
    gmap = [0] * sum(sizes)
    pos = 0
    for grp, s in enumerate(sizes):
        for h in perm[pos:pos + s]:
            gmap[int(h)] = grp
        pos += s
    return tuple(gmap)


SMALL = {
    # MHA with a singleton, odd ranks, a 1-token and an empty sequence, shuffled pages
    "mha_odd": dict(hidden=256, num_q_heads=8, num_kv_heads=8, head_dim=64, sizes=(1, 3, 4),
                    group_rank=(37, 101, 129), value_rank=96, seq_lens=(300, 64, 1, 0, 129),
                    permute_pages=True, split=128),
    # GQA 4 queries per KV head, uneven groups
    "gqa_uneven": dict(hidden=512, num_q_heads=16, num_kv_heads=4, head_dim=128, sizes=(2, 1, 1),
                       group_rank=(200, 77, 128), value_rank=256, seq_lens=(1000, 777),
                       permute_pages=False, split=256),
    # one group holding every head, value rank not a multiple of 64
    "single_group": dict(hidden=384, num_q_heads=4, num_kv_heads=4, head_dim=64, sizes=(4,),
                         group_rank=(160,), value_rank=200, seq_lens=(517,), permute_pages=True,
                         split=64),
    # many singletons (as the grouping often yields), d_h 128
    "singletons": dict(hidden=1024, num_q_heads=8, num_kv_heads=8, head_dim=128,
                       sizes=(1, 1, 1, 2, 1, 1, 1), group_rank=(31, 64, 17, 150, 99, 128, 5),
                       value_rank=384, seq_lens=(2049, 65, 640), permute_pages=True, split=512),
    # 32 heads with two 16-head tiles and odd group boundaries inside tiles
    "mha32_two_tiles": dict(hidden=1024, num_q_heads=32, num_kv_heads=32, head_dim=64,
                            sizes=(7, 9, 5, 1, 10), group_rank=(201, 333, 97, 31, 160),
                            value_rank=512, seq_lens=(700, 1, 64, 383), permute_pages=True,
                            split=256),
    # value rank above what the MFMA accumulators hold: the portable bf16 kernels run
    "valu_bf16": dict(hidden=2560, num_q_heads=32, num_kv_heads=32, head_dim=128,
                      sizes=(8, 8, 8, 8), group_rank=(300, 200, 100, 50), value_rank=2304,
                      seq_lens=(200, 70), permute_pages=False, split=128),
    # 40 rows a KV head and value rank 1024: the eight-wave up-projection
    "rows40_rv1024": dict(hidden=1024, num_q_heads=8, num_kv_heads=8, head_dim=128, sizes=(3, 5),
                          group_rank=(64, 100), value_rank=1024,
                          seq_lens=tuple((13 * i + 1) % 90 for i in range(40)),
                          permute_pages=False, split=64),
    # head size 96: the per-sequence query fold and the narrow up-projections
    "head96": dict(hidden=384, num_q_heads=8, num_kv_heads=4, head_dim=96, sizes=(1, 3),
                   group_rank=(50, 130), value_rank=144, seq_lens=(250, 3, 70),
                   permute_pages=True, split=64),
    # more sequences than the query fold stages at once (64), short and
    # empty ones among them, and more than 64 rows a KV head
    "many_seqs": dict(hidden=512, num_q_heads=8, num_kv_heads=8, head_dim=64, sizes=(3, 5),
                      group_rank=(96, 40), value_rank=128,
                      seq_lens=tuple((37 * i) % 201 for i in range(70)), permute_pages=True,
                      split=64),
    # groups of 8, 12 and 12 rows: the plan cuts the smallest group, so one
    # 16-row tile loads two separate ranges of key chunks
    "gqa_reordered": dict(hidden=512, num_q_heads=32, num_kv_heads=8, head_dim=64, sizes=(2, 3, 3),
                          group_rank=(96, 128, 160), value_rank=256, seq_lens=(900, 300, 65),
                          permute_pages=True, split=256),
}


def _small_inputs(name, dtype="bf16"):
    c = SMALL[name]
    wl = custom_workload(name=name, seed=100 + list(SMALL).index(name), hidden=c["hidden"],
                         num_q_heads=c["num_q_heads"], num_kv_heads=c["num_kv_heads"],
                         head_dim=c["head_dim"], group_of_kv=_groups(c["sizes"], 7),
                         group_rank=c["group_rank"], value_rank=c["value_rank"], dtype=dtype,
                         batch=len(c["seq_lens"]), seq_lens=c["seq_lens"],
                         prefill_lens=c["seq_lens"], factor_scheme="orthonormal",
                         permute_pages=c["permute_pages"])
    return wl, make_inputs(wl), c["split"]


def _all_rows(inp, q=None):
    wl = inp.wl
    pairs = [(b, h) for b in range(wl.batch) for h in range(wl.num_q_heads)]
    return oracle_rows(inp, pairs, q=q)


# ------------------------------------------------------------------ tiny fp32
def test_tiny_mha_f32_append_then_decode():
    wl = make_workload("tiny_mha_f32")
    inp = make_inputs(wl)
    plan = plan_for(wl)
    pool = gpu_pool_with_append(inp, plan)
    got_pool = pool.cpu().numpy()
    # append: every latent within fp32 rounding of the exact product
    Zk_g, Zv_g = olayout.unpack(got_pool, inp.page_table, 0, 256, wl.key_rank_total, wl.value_rank)
    for Zg, L in ((Zk_g, inp.L_keys), (Zv_g, inp.L_value)):
        exact = oappend.down_project(inp.x, L)
        bound = wl.hidden * 2.0 ** -24 * oappend.abs_bound(inp.x, L) + np.abs(exact) * 2.0 ** -23
        assert np.all(np.abs(Zg - exact) <= bound)
    out = run_decode(inp, plan, pool)
    ref_pool = oracle_pool(inp)
    ref = oattn.decode(inp.q, ref_pool, inp.page_table, wl.seq_lens, inp.R_blocks, inp.R_value,
                       book_for(wl), chunk=None)
    errs = [row_rel_err(out[0, h], ref[0, h]) for h in range(wl.num_q_heads)]
    _report("tiny_mha_f32", errs)
    assert max(errs) <= TOL_REL_ROW_F32


# ------------------------------------------------------------------ small bf16
@pytest.mark.parametrize("name", list(SMALL))
def test_small_decode_all_rows(name):
    wl, inp, split = _small_inputs(name)
    plan = plan_for(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    ref = _all_rows(inp)
    errs = []
    for (b, h), o in ref.items():
        if wl.seq_lens[b] == 0:
            assert np.all(out[b, h] == 0)
            continue
        errs.append(row_rel_err(out[b, h], o))
    _report(name, errs)
    assert max(errs) <= TOL_REL_ROW


# (case, decode_waves, head_slices): launch shapes of the MFMA decode beyond
# the defaults -- 4 and 8 waves, one and two 16-head tiles, all key block sizes,
# value-tile capacities 6, 8 and 32 -- each checked on every row
LAUNCH_SHAPES = [("gqa_uneven", 4, 0), ("gqa_uneven", 8, 2), ("singletons", 4, 0),
                 ("mha32_two_tiles", 4, 0), ("mha32_two_tiles", 4, 2), ("valu_bf16", 8, 2),
                 ("single_group", 4, 0), ("gqa_reordered", 4, 0)]


@pytest.mark.parametrize("name, waves, slices", LAUNCH_SHAPES)
def test_decode_launch_shapes(name, waves, slices):
    from paper_2607_24331_amd import Plan
    wl, inp, split = _small_inputs(name)
    plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, split, slices, waves)
    geo = plan.geometry
    assert geo["mfma_path"] == 1 and geo["decode_waves"] == waves
    print(f"[shape] {name} waves {waves} slices {geo['head_slices']} ring {geo['decode_ring']} "
          f"tiles/wave {geo['value_tiles_per_wave']}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    ref = _all_rows(inp)
    errs = []
    for (b, h), o in ref.items():
        if wl.seq_lens[b] == 0:
            assert np.all(out[b, h] == 0)
            continue
        errs.append(row_rel_err(out[b, h], o))
    _report(f"{name}/w{waves}/j{slices}", errs)
    assert max(errs) <= TOL_REL_ROW


def test_launch_shapes_cover_both_rings():
    from paper_2607_24331_amd import Plan
    rings, caps = set(), set()
    for name, waves, slices in LAUNCH_SHAPES:
        wl, _, split = _small_inputs(name)
        geo = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                   wl.group_rank, wl.value_rank, wl.dtype, split, slices, waves).geometry
        rings.add(geo["decode_ring"])
        caps.add(geo["value_tiles_per_wave"])
    assert rings == {12, 14, 16}
    assert max(caps) > 16 and min(caps) <= 6


# (case, Q, latent dtype): several causal queries a sequence.  mha_odd holds
# a one-token and an empty sequence (queries that see nothing give zeros);
# 32 heads x 8 queries fill all eight row slices of the MFMA path; f32 runs
# the portable kernels.
MULTI = [("gqa_uneven", 4, "bf16"), ("mha32_two_tiles", 2, "bf16"), ("mha32_two_tiles", 8, "bf16"),
         ("mha_odd", 8, "bf16"), ("singletons", 3, "bf16"), ("mha_odd", 3, "f32"),
         ("many_seqs", 2, "bf16")]


@pytest.mark.parametrize("name, Q, dtype", MULTI)
def test_multi_query_all_rows(name, Q, dtype):
    from paper_2607_24331_amd import Plan, decode
    wl, inp, split = _small_inputs(name, dtype)
    plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, split, queries_per_seq=Q)
    geo = plan.geometry
    assert geo["queries_per_seq"] == Q
    assert geo["mfma_path"] == (1 if dtype == "bf16" else 0)
    print(f"[multi] {name} Q {Q} {dtype} slices {geo['head_slices']}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    qm = np.random.default_rng(11).standard_normal(
        (wl.batch, Q, wl.num_q_heads, wl.head_dim)).astype(np.float32)
    out = decode(plan, torch.from_numpy(qm).cuda(), pool, torch.from_numpy(inp.page_table).cuda(),
                 torch.from_numpy(inp.seq_lens).cuda(), int(max(wl.seq_lens)),
                 dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype))
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = oattn.decode_multi(qm, oracle_pool(inp), inp.page_table, wl.seq_lens, inp.R_blocks,
                             inp.R_value, book_for(wl), chunk=None)
    errs = []
    for b in range(wl.batch):
        for i in range(Q):
            seen = oattn.visible_tokens(wl.seq_lens[b], Q, i)
            for h in range(wl.num_q_heads):
                if seen == 0:
                    assert np.all(got[b, i, h] == 0)
                else:
                    errs.append(row_rel_err(got[b, i, h], ref[b, i, h]))
    _report(f"multi/{name}/Q{Q}/{dtype}", errs)
    assert max(errs) <= (TOL_REL_ROW if dtype == "bf16" else TOL_REL_ROW_F32)


def test_peaked_softmax():
    wl, inp, split = _small_inputs("gqa_uneven")
    plan = plan_for(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    q = inp.q * 16.0
    out = run_decode(inp, plan, pool, q=q)
    ref = _all_rows(inp, q=q)
    errs = [row_rel_err(out[b, h], o) for (b, h), o in ref.items()]
    _report("peaked", errs)
    assert max(errs) <= TOL_REL_ROW


def test_split_invariance_and_determinism():
    wl, inp, _ = _small_inputs("singletons")
    outs = []
    for split in (64, 192, 1024, 4096):
        plan = plan_for(wl, split)
        pool = gpu_pool_with_append(inp, plan)
        a = run_decode(inp, plan, pool)
        b = run_decode(inp, plan, pool)
        assert np.array_equal(a, b)                       # bitwise repeatable
        outs.append(a)
    for o in outs[1:]:
        assert np.max(np.abs(o - outs[0])) <= 1e-3 * np.max(np.abs(outs[0]))


def test_physical_page_permutation_is_invisible():
    wl, inp, split = _small_inputs("mha_odd")
    plan = plan_for(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    # move every page to a new physical place and rewrite the table
    g = np.random.default_rng(3)
    perm = g.permutation(inp.num_pages)
    pool2 = torch.empty_like(pool)
    pool2[torch.from_numpy(perm).cuda()] = pool
    table2 = perm[inp.page_table].astype(np.int32)
    inp.page_table = table2
    out2 = run_decode(inp, plan, pool2)
    assert np.array_equal(out, out2)


def test_out_of_range_pages_are_skipped_without_fault():
    wl, inp, split = _small_inputs("gqa_uneven")
    plan = plan_for(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    inp.page_table = inp.page_table.copy()
    inp.page_table[1, 3] = inp.num_pages + 5      # invalid entry inside sequence 1
    out = run_decode(inp, plan, pool)
    assert np.isfinite(out).all()


# --------------------------------------------------------------- append checks
def test_append_layout_bit_exact_on_exact_inputs():
    # Small-integer x and L: every product and sum is exact in fp32 and bf16,
    # so the pool must equal the oracle's packing bit for bit, including the
    # zero padding columns and the untouched slots.
    wl, inp, split = _small_inputs("singletons")
    g = np.random.default_rng(9)
    n = 150
    x = g.integers(-2, 3, size=(n, wl.hidden)).astype(np.float32) * (g.random((n, wl.hidden)) < 0.02)
    Lk = g.integers(-2, 3, size=(wl.hidden, wl.key_rank_total)).astype(np.float32)
    Lv = g.integers(-2, 3, size=(wl.hidden, wl.value_rank)).astype(np.float32)
    pages = 5
    table = np.array([[4, 0, 2]], dtype=np.int32)
    start = 37
    pos = start + np.arange(n)
    slots = table[0, pos // 64].astype(np.int64) * 64 + pos % 64
    sentinel = np.float32(-7.0)
    ref = np.full((pages, olayout.page_elems(wl.key_rank_total, wl.value_rank)), sentinel, np.float32)
    oappend.append(ref, table, 0, start, x, Lk, Lv, "bf16")
    # the padding key columns of written slots are zero
    RK, RKp = wl.key_rank_total, olayout.key_width_padded(wl.key_rank_total)
    for p in pos:
        ref[table[0, p // 64], olayout.key_offset(p % 64, np.arange(RK, RKp), RK)] = 0
    plan = plan_for(wl, split)
    from paper_2607_24331_amd import latent_append
    pool = dev(np.full(ref.shape, sentinel, np.float32), "bf16")
    latent_append(plan, dev(x, "bf16"), dev(Lk.T, "bf16"), dev(Lv.T, "bf16"),
                  torch.from_numpy(slots).cuda(), pool)
    torch.cuda.synchronize()
    got_bits = pool.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got_bits, bf16_bits_from_f32(ref.astype(np.float32)))


def test_append_random_within_one_ulp():
    wl, inp, split = _small_inputs("gqa_uneven")
    g = np.random.default_rng(1)
    n = 333
    from workloads.inputs import to_storage
    x = to_storage(g.standard_normal((n, wl.hidden)), "bf16")
    Lk = to_storage(g.standard_normal((wl.hidden, wl.key_rank_total)) / np.sqrt(wl.hidden), "bf16")
    Lv = to_storage(g.standard_normal((wl.hidden, wl.value_rank)) / np.sqrt(wl.hidden), "bf16")
    table = np.arange(6, dtype=np.int32)[None, :]
    slots = np.arange(n, dtype=np.int64)
    slots[5] = -1                       # skipped token
    plan = plan_for(wl, split)
    from paper_2607_24331_amd import latent_append
    pool = plan.new_pool(6)
    latent_append(plan, dev(x, "bf16"), dev(Lk.T, "bf16"), dev(Lv.T, "bf16"),
                  torch.from_numpy(slots).cuda(), pool)
    torch.cuda.synchronize()
    Zk_g, Zv_g = olayout.unpack(pool.float().cpu().numpy(), table, 0, n, wl.key_rank_total, wl.value_rank)
    for Zg, L in ((Zk_g, Lk), (Zv_g, Lv)):
        exact = oappend.down_project(x, L)
        rounded = obf16.round_to_bf16(exact)
        bound = obf16.ulp_bf16(rounded) + wl.hidden * 2.0 ** -24 * oappend.abs_bound(x, L)
        diff = np.abs(Zg - rounded)
        keep = np.ones(n, bool)
        keep[5] = False
        assert np.all(diff[keep] <= bound[keep])
        assert np.mean(Zg[keep] == rounded[keep]) > 0.99
        assert np.all(Zg[5] == 0)        # skipped slot untouched


# ------------------------------------------------------------ full workloads
@pytest.mark.parametrize("name", [n for n in WORKLOAD_NAMES if n != "tiny_mha_f32"])
def test_full_workload_sampled_rows(name):
    wl = make_workload(name)
    print(f"[parity] start {name}", flush=True)
    inp = make_inputs(wl)
    plan = plan_for(wl)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    assert np.isfinite(out).all()
    out2 = run_decode(inp, plan, pool)
    assert np.array_equal(out, out2)
    if wl.append_tokens:
        # the appended latents, read back through the oracle's layout
        RK, rv = wl.key_rank_total, wl.value_rank
        first = wl.prefill_lens[0] // 64
        last = -(-wl.seq_lens[0] // 64)
        pages = torch.from_numpy(inp.page_table[0, first:last].astype(np.int64)).cuda()
        part = pool[pages].float().cpu().numpy()
        tbl = np.arange(part.shape[0], dtype=np.int32)[None, :]
        skip = wl.prefill_lens[0] % 64
        Zk_g, Zv_g = olayout.unpack(part, tbl, 0, skip + wl.append_tokens, RK, rv)
        for Zg, L in ((Zk_g[skip:], inp.L_keys), (Zv_g[skip:], inp.L_value)):
            exact = oappend.down_project(inp.x, L)
            rounded = obf16.round_to_bf16(exact)
            bound = obf16.ulp_bf16(rounded) + wl.hidden * 2.0 ** -24 * oappend.abs_bound(inp.x, L)
            assert np.all(np.abs(Zg - rounded) <= bound)
    if wl.batch >= 32:
        pairs = every_sequence_pairs(wl)         # one head of every sequence, every group
    else:
        pairs = sample_pairs(wl, 8 if wl.seq_lens[0] < 100000 else 5)
    ref = oracle_rows(inp, pairs)
    errs = [row_rel_err(out[b, h], ref[(b, h)]) for b, h in pairs]
    _report(name, errs)
    assert max(errs) <= TOL_REL_ROW


def test_long_split_list_deep_batch_merge():
    # 128 splits of 64 tokens over 16 sequences and value rank 1024: the
    # merge for long split lists with sixteen value ranks a work-group
    wl = custom_workload(name="deep_long", seed=91, hidden=1024, num_q_heads=8, num_kv_heads=8,
                         head_dim=128, group_of_kv=(0, 0, 0, 1, 1, 1, 1, 1),
                         group_rank=(96, 160), value_rank=1024, dtype="bf16", batch=16,
                         seq_lens=tuple(8192 - 517 * (i % 5) for i in range(16)),
                         factor_scheme="orthonormal")
    inp = make_inputs(wl)
    plan = plan_for(wl, 64)
    info = plan.launch_info(wl.batch, max(wl.seq_lens))
    assert info["split_tokens"] == 64
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    assert np.array_equal(out, run_decode(inp, plan, pool))
    pairs = sample_pairs(wl, 8)
    ref = oracle_rows(inp, pairs)
    errs = [row_rel_err(out[b, h], ref[(b, h)]) for b, h in pairs]
    _report("deep_long", errs)
    assert max(errs) <= TOL_REL_ROW


def test_wide_up_projection_tiles_many_rows():
    # 70 rows over 32 KV heads of 128 (two 64-row groups a head): the grid
    # holds 256 (KV head, row group, 32-column tile) work-groups, so the MFMA
    # up-projection takes 32-column tiles; every row checked
    wl = custom_workload(name="mha32_b70", seed=92, hidden=4096, num_q_heads=32, num_kv_heads=32,
                         head_dim=128, group_of_kv=tuple(i // 8 for i in range(32)),
                         group_rank=(64, 96, 40, 72), value_rank=256, dtype="bf16", batch=70,
                         seq_lens=tuple(1 + (29 * i) % 150 for i in range(70)),
                         factor_scheme="orthonormal")
    inp = make_inputs(wl)
    plan = plan_for(wl)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    ref = _all_rows(inp)
    errs = [row_rel_err(out[b, h], o) for (b, h), o in ref.items()]
    _report("mha32_b70", errs)
    assert max(errs) <= TOL_REL_ROW


def every_sequence_pairs(wl):
    """One (sequence, head) row of every sequence; sequence b takes a head of
    group b mod G (the group's heads in turn), so every group is covered."""
    qpk = wl.num_q_heads // wl.num_kv_heads
    members = [[kv for kv in range(wl.num_kv_heads) if wl.group_of_kv[kv] == g]
               for g in range(wl.num_groups)]
    pairs = []
    for b in range(wl.batch):
        g = b % wl.num_groups
        kv = members[g][(b // wl.num_groups) % len(members[g])]
        pairs.append((b, kv * qpk + (b % qpk)))
    assert {wl.group_of_kv[h // qpk] for _, h in pairs} == set(range(wl.num_groups))
    return pairs


@pytest.mark.parametrize("passes", [1, 0])
def test_multi_query_long_layer_benchmarked_shape(passes):
    # the long-context layer with 4 causal queries a sequence, in the launch
    # shapes the benchmark times: the single-pass kernel (4 row slices,
    # 2048-token splits), and the default, the two-pass kernels (the 4 slices
    # sharing one walk over the value latents); rows of two heads (different
    # groups) for every query, query 0 included
    from paper_2607_24331_amd import Plan, decode
    wl = make_workload("mha_long_t128k")
    print(f"[parity] start mha_long_t128k Q=4 passes {passes}", flush=True)
    inp = make_inputs(wl)
    Q = 4
    plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, 2048 if passes == 1 else 0,
                queries_per_seq=Q, decode_passes=passes)
    geo = plan.geometry
    assert geo["mfma_path"] == 1 and geo["head_slices"] == 4
    info = plan.launch_info(wl.batch, int(max(wl.seq_lens)))
    assert info["kernels"] == (1 if passes == 1 else 2) and info["head_slices"] == 4, info
    pool = gpu_pool_with_append(inp, plan)
    qm = np.random.default_rng(12).standard_normal(
        (wl.batch, Q, wl.num_q_heads, wl.head_dim)).astype(np.float32)
    out = decode(plan, torch.from_numpy(qm).cuda(), pool, torch.from_numpy(inp.page_table).cuda(),
                 torch.from_numpy(inp.seq_lens).cuda(), int(max(wl.seq_lens)),
                 dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype))
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all()
    from gpu_common import seq_latents
    bk = book_for(wl)
    Zk, Zv = seq_latents(inp, 0)
    T = wl.seq_lens[0]
    heads = sample_pairs(wl, 2, seed=4)[:2]
    errs = []
    for _, h in heads:
        K, V = oattn.rebuild(Zk, Zv, inp.R_blocks, inp.R_value, bk, h)   # once a head
        for i in range(Q):
            n = oattn.visible_tokens(T, Q, i)
            ref = oattn.attend(qm[0, i, h], K[:n], V[:n])
            errs.append(row_rel_err(got[0, i, h], ref))
        del K, V
    _report(f"mha_long_t128k/Q4/{'single' if passes == 1 else 'two'}-pass", errs)
    assert max(errs) <= TOL_REL_ROW


def test_value_rank_3072_full_layer_both_kernel_sets():
    # a full-size MHA layer (4 x 32768 tokens) with value rank 3072: the
    # single-pass kernel needs two row slices, the two-pass kernels one
    from paper_2607_24331_amd import Plan
    wl = custom_workload(name="mha_rv3072_b4_t32k", seed=3072, hidden=4096, num_q_heads=32,
                         num_kv_heads=32, head_dim=128, group_of_kv=_groups((8, 6, 6, 5, 4, 3), 5),
                         group_rank=(400, 300, 300, 240, 200, 96), value_rank=3072, dtype="bf16",
                         batch=4, seq_lens=(32768, 32768, 30000, 32768),
                         prefill_lens=(32768, 32768, 30000, 32768), factor_scheme="orthonormal")
    print("[parity] start mha_rv3072_b4_t32k", flush=True)
    inp = make_inputs(wl)
    pairs = sample_pairs(wl, 6, seed=9)
    ref = oracle_rows(inp, pairs)
    outs = []
    for passes in (1, 0):
        plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                    wl.group_rank, wl.value_rank, wl.dtype, decode_passes=passes)
        geo = plan.geometry
        assert geo["mfma_path"] == 1 and geo["head_slices"] == 2
        pool = gpu_pool_with_append(inp, plan)
        out = run_decode(inp, plan, pool)
        assert np.isfinite(out).all()
        errs = [row_rel_err(out[b, h], ref[(b, h)]) for b, h in pairs]
        _report(f"mha_rv3072/{'single-pass' if passes == 1 else 'default (two-pass)'}", errs)
        assert max(errs) <= TOL_REL_ROW
        outs.append(out)
        del pool
    assert np.max(np.abs(outs[0] - outs[1])) <= 1e-2 * np.max(np.abs(outs[0]))


@pytest.mark.parametrize("n", [1, 129, 640])
def test_append_mfma_ragged_token_counts_reproducible(n):
    # one token, one past a 128-token tile, and five full tiles through the
    # MFMA kernel (hidden 512: eight 64-deep stages, four stage buffers): each
    # latent within one bf16 ulp of the rounded exact product, and a second
    # call writes the same bits
    hidden = 512
    wl = custom_workload(name="append_n", seed=78, hidden=hidden, num_q_heads=4, num_kv_heads=4,
                         head_dim=64, group_of_kv=(0, 1, 1, 0), group_rank=(50, 61), value_rank=100,
                         dtype="bf16", batch=1, seq_lens=(n,), prefill_lens=(n,))
    g = np.random.default_rng(n)
    from workloads.inputs import to_storage
    x = to_storage(g.standard_normal((n, hidden)), "bf16")
    Lk = to_storage(g.standard_normal((hidden, 111)) / np.sqrt(hidden), "bf16")
    Lv = to_storage(g.standard_normal((hidden, 100)) / np.sqrt(hidden), "bf16")
    npages = (n + 63) // 64
    table = np.arange(npages, dtype=np.int32)[None, :]
    slots = np.arange(n, dtype=np.int64)
    plan = plan_for(wl)
    from paper_2607_24331_amd import latent_append
    pools = []
    for _ in range(2):
        pool = plan.new_pool(npages)
        latent_append(plan, dev(x, "bf16"), dev(Lk.T, "bf16"), dev(Lv.T, "bf16"),
                      torch.from_numpy(slots).cuda(), pool)
        torch.cuda.synchronize()
        pools.append(pool.view(torch.int16).cpu().numpy().copy())
        last = pool
    assert np.array_equal(pools[0], pools[1])
    Zk_g, Zv_g = olayout.unpack(last.float().cpu().numpy(), table, 0, n, 111, 100)
    for Zg, L in ((Zk_g, Lk), (Zv_g, Lv)):
        exact = oappend.down_project(x, L)
        rounded = obf16.round_to_bf16(exact)
        bound = obf16.ulp_bf16(rounded) + hidden * 2.0 ** -24 * oappend.abs_bound(x, L)
        assert np.all(np.abs(Zg - rounded) <= bound)


@pytest.mark.parametrize("hidden", [200, 320, 384, 512])
def test_append_bf16_both_kernels(hidden):
    # hidden 200 (not a multiple of 64) takes the portable kernel; 320, 384
    # and 512 the MFMA one with 1, 2 and 4 k stages in flight
    wl = custom_workload(name="append_h", seed=77, hidden=hidden, num_q_heads=4, num_kv_heads=4,
                         head_dim=64, group_of_kv=(0, 1, 1, 0), group_rank=(50, 61), value_rank=100,
                         dtype="bf16", batch=1, seq_lens=(130,), prefill_lens=(130,))
    g = np.random.default_rng(5)
    from workloads.inputs import to_storage
    n = 130
    x = to_storage(g.standard_normal((n, hidden)), "bf16")
    Lk = to_storage(g.standard_normal((hidden, 111)) / np.sqrt(hidden), "bf16")
    Lv = to_storage(g.standard_normal((hidden, 100)) / np.sqrt(hidden), "bf16")
    perm = np.random.default_rng(6).permutation(3).astype(np.int32)
    table = perm[None, :]
    pos = np.arange(n)
    slots = table[0, pos // 64].astype(np.int64) * 64 + pos % 64
    plan = plan_for(wl)
    from paper_2607_24331_amd import latent_append
    pool = plan.new_pool(3)
    latent_append(plan, dev(x, "bf16"), dev(Lk.T, "bf16"), dev(Lv.T, "bf16"),
                  torch.from_numpy(slots).cuda(), pool)
    torch.cuda.synchronize()
    Zk_g, Zv_g = olayout.unpack(pool.float().cpu().numpy(), table, 0, n, 111, 100)
    for Zg, L in ((Zk_g, Lk), (Zv_g, Lv)):
        exact = oappend.down_project(x, L)
        rounded = obf16.round_to_bf16(exact)
        bound = obf16.ulp_bf16(rounded) + hidden * 2.0 ** -24 * oappend.abs_bound(x, L)
        assert np.all(np.abs(Zg - rounded) <= bound)
        assert np.mean(Zg == rounded) > 0.99
