"""Host-side checks of libdckv: exported symbols, plan bookkeeping against the
oracle's independent bookkeeping (bit-exact), and validation errors.  Nothing
here launches a kernel."""

import ctypes

import numpy as np
import pytest
import torch

from oracle import layout as olayout
from oracle.bookkeeping import book_for, make_book
from workloads import WORKLOAD_NAMES, make_workload

capi = pytest.importorskip("paper_2607_24331_amd.capi")


@pytest.fixture(scope="module")
def lib():
    return capi.load()


def test_every_declared_function_is_exported(lib):
    names = capi.header_functions()
    assert set(names) == set(capi.SIGNATURES), names
    for name in names:
        assert hasattr(lib, name), name


def _plan(wl, split_tokens=0):
    from paper_2607_24331_amd import Plan
    return Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, split_tokens)


@pytest.mark.parametrize("name", WORKLOAD_NAMES)
def test_bookkeeping_matches_oracle(name):
    wl = make_workload(name)
    bk = book_for(wl)
    info = _plan(wl).info()
    geo = info["geometry"]
    assert info["koff"] == bk.koff
    assert info["pos_in_group"] == bk.pos_in_group
    assert info["qoff"] == bk.qoff
    assert info["roff"] == bk.roff
    assert geo["key_rank_total"] == bk.key_rank_total
    assert geo["key_width_padded"] == olayout.key_width_padded(bk.key_rank_total)
    assert geo["value_width_padded"] == olayout.value_width_padded(bk.value_rank)
    assert geo["page_elems"] == olayout.page_elems(bk.key_rank_total, bk.value_rank)
    assert geo["value_base"] == olayout.value_base(bk.key_rank_total)
    assert geo["q_per_kv"] == bk.q_per_kv
    assert geo["folded_query_len"] == bk.qoff[-1]
    assert geo["key_factor_elems"] == bk.roff[-1]


def test_bookkeeping_random_layers():
    from paper_2607_24331_amd import Plan
    g = np.random.default_rng(5)
    for _ in range(200):
        Hkv = int(g.integers(1, 17))
        qpk = int(g.choice([1, 2, 4]))
        if Hkv * qpk > 64:
            continue
        d = int(g.choice([8, 64, 128]))
        G = int(g.integers(1, Hkv + 1))
        gmap = list(g.permutation(np.concatenate([np.arange(G), g.integers(0, G, Hkv - G)])))
        m = int(g.integers(64, 5000))
        sizes = [gmap.count(i) for i in range(G)]
        ranks = [int(g.integers(1, min(m, s * d) + 1)) for s in sizes]
        rv = int(g.integers(1, min(m, Hkv * d, 4096) + 1))
        if max(ranks) > 4096:
            continue
        bk = make_book(m, Hkv * qpk, Hkv, d, gmap, ranks, rv)
        info = Plan(m, Hkv * qpk, Hkv, d, gmap, ranks, rv, "bf16").info()
        assert (info["koff"], info["pos_in_group"], info["qoff"], info["roff"]) == \
            (bk.koff, bk.pos_in_group, bk.qoff, bk.roff)


@pytest.mark.parametrize("change, status", [
    (dict(gmap=[0, 0, 0, 0]), "DCKV_EINVAL"),            # group 1 empty
    (dict(gmap=[0, 1, 2, 1]), "DCKV_EINVAL"),            # group id out of range
    (dict(ranks=[0, 8]), "DCKV_EINVAL"),
    (dict(ranks=[33, 8]), "DCKV_EINVAL"),                # above h_g * d_h = 32
    (dict(num_q=6), "DCKV_EINVAL"),
    (dict(value_rank=65), "DCKV_EINVAL"),
    (dict(dtype=7), "DCKV_EDTYPE"),
    (dict(split=100), "DCKV_EINVAL"),
    (dict(head_dim=300), "DCKV_EINVAL"),
    (dict(queries=65), "DCKV_EINVAL"),                 # above DCKV_MAX_QUERIES
    (dict(queries=-1), "DCKV_EINVAL"),
])
def test_plan_create_rejects(lib, change, status):
    a = dict(hidden=64, num_q=4, gmap=[0, 1, 0, 1], ranks=[8, 8], value_rank=16, dtype=1, split=0,
             head_dim=16, queries=0)
    a.update(change)
    gm = (ctypes.c_int32 * 4)(*a["gmap"])
    rk = (ctypes.c_int32 * 2)(*a["ranks"])
    desc = capi.LayerDesc(a["hidden"], a["num_q"], 4, a["head_dim"], 2,
                          ctypes.cast(gm, ctypes.POINTER(ctypes.c_int32)),
                          ctypes.cast(rk, ctypes.POINTER(ctypes.c_int32)),
                          a["value_rank"], a["dtype"], a["split"], 0, a["queries"])
    out = ctypes.c_void_p(12345)
    st = lib.dckv_plan_create(ctypes.byref(desc), ctypes.byref(out))
    assert capi.STATUS_NAMES[st] == status
    assert out.value == 12345                       # untouched on failure
    assert lib.dckv_last_error().decode().startswith("plan_create:")


def test_workspace_bytes_grows_with_work():
    from paper_2607_24331_amd import Plan
    wl = make_workload("gqa8b_b4_t32k")
    for passes in (1, 2):                 # either kernel set, chosen for every call
        p = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                 wl.group_rank, wl.value_rank, wl.dtype, decode_passes=passes)
        a = p.workspace_bytes(4, 32768)
        assert a > p.workspace_bytes(1, 32768) > 0
        assert a >= p.workspace_bytes(4, 1024)
        assert p.workspace_bytes(4, 0) > 0


@pytest.mark.skipif(torch.cuda.is_available(), reason="raw fake pointers are only passed on a host without a GPU")
def test_call_validation_never_launches(lib):
    wl = make_workload("tiny_mha_f32")
    p = _plan(wl)
    h = p.handle
    A = 1 << 20                                       # aligned fake address, never dereferenced
    # append: null pointer, misalignment, bad sizes
    assert lib.dckv_latent_append(h, None, 4, A, A, A, A, 4, None) == capi.DCKV_EINVAL
    assert lib.dckv_latent_append(h, A + 2, 4, A, A, A, A, 4, None) == capi.DCKV_EALIGN
    assert lib.dckv_latent_append(h, A, -1, A, A, A, A, 4, None) == capi.DCKV_EINVAL
    assert lib.dckv_latent_append(h, A, 4, A, A, A, A, 0, None) == capi.DCKV_EINVAL
    assert lib.dckv_latent_append(h, None, 0, None, None, None, None, 0, None) == capi.DCKV_OK
    # decode
    ws_need = p.workspace_bytes(1, 256)
    args = [h, A, 1, A, 4, A, 4, A, 256, A, A, A, A, ws_need, None]

    def call(**kw):
        a = list(args)
        idx = {"q": 1, "batch": 2, "pool": 3, "num_pages": 4, "table": 5, "max_pages": 6,
               "lens": 7, "max_context": 8, "rk": 9, "rv": 10, "out": 11, "ws": 12, "ws_bytes": 13}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.dckv_decode(*a)
    assert call(q=None) == capi.DCKV_EINVAL
    assert call(max_context=257) == capi.DCKV_EINVAL          # beyond max_pages * 64
    assert call(max_context=-1) == capi.DCKV_EINVAL
    assert call(num_pages=0) == capi.DCKV_EINVAL
    assert call(max_pages=0) == capi.DCKV_EINVAL
    assert call(batch=-2) == capi.DCKV_EINVAL
    assert call(out=A + 4) == capi.DCKV_EALIGN
    assert call(ws=A + 16) == capi.DCKV_EALIGN
    assert call(ws_bytes=ws_need - 1) == capi.DCKV_EWORKSPACE
    assert "workspace" in lib.dckv_last_error().decode()
    assert call(batch=0) == capi.DCKV_OK                      # no-op


@pytest.mark.skipif(torch.cuda.is_available(), reason="raw fake pointers are only passed on a host without a GPU")
def test_noalloc_validation_never_launches(lib):
    # the decode without a workspace: the same argument checks, then the
    # scratch bound (64-token splits over 131072 tokens need far more than
    # the fixed array), all before any HIP call
    from paper_2607_24331_amd import Plan
    wl = make_workload("gqa8b_b4_t32k")
    p = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv, wl.group_rank,
             wl.value_rank, wl.dtype, 64)
    A = 1 << 20
    args = [p.handle, A, 1, A, 4096, A, 2048, A, 131072, A, A, A, None]
    assert p.workspace_bytes(1, 131072) > capi.NOALLOC_SCRATCH_BYTES
    assert lib.dckv_decode_noalloc(*args) == capi.DCKV_EWORKSPACE
    assert "scratch" in lib.dckv_last_error().decode()
    bad = list(args)
    bad[1] = None
    assert lib.dckv_decode_noalloc(*bad) == capi.DCKV_EINVAL
    bad = list(args)
    bad[11] = A + 4
    assert lib.dckv_decode_noalloc(*bad) == capi.DCKV_EALIGN
    bad = list(args)
    bad[2] = 0
    assert lib.dckv_decode_noalloc(*bad) == capi.DCKV_OK      # batch 0: no-op
    assert lib.dckv_decode_noalloc(None, *args[1:]) == capi.DCKV_EINVAL


def test_binding_rejects_host_tensors():
    from paper_2607_24331_amd import decode, latent_append
    wl = make_workload("tiny_mha_f32")
    p = _plan(wl)
    x = torch.zeros(4, 512)
    with pytest.raises(ValueError, match="GPU"):
        latent_append(p, x, torch.zeros(512, 128), torch.zeros(512, 128),
                      torch.zeros(4, dtype=torch.int64), torch.zeros(4, p.page_elems))
    with pytest.raises(ValueError, match="GPU"):
        decode(p, torch.zeros(1, 8, 64), torch.zeros(4, p.page_elems), torch.zeros(1, 4, dtype=torch.int32),
               torch.zeros(1, dtype=torch.int32), 256, torch.zeros(p.key_factor_elems),
               torch.zeros(128, 512))


def test_decode_path_selection():
    expect = {"tiny_mha_f32": 0, "mha7b_b8_t4k": 1, "gqa8b_b4_t32k": 1, "mha_long_t128k": 1,
              "mha_ragged_b64": 1}
    for name, mfma in expect.items():
        assert _plan(make_workload(name)).geometry["mfma_path"] == mfma, name
    from paper_2607_24331_amd import Plan
    # value rank 2304 with 32 heads: the two-pass kernels take any value rank;
    # the single-pass kernel takes two slices of 16 rows (its accumulators
    # hold 2304 ranks for 16 rows a slice, not 32)
    args = (2560, 32, 32, 128, [i // 8 for i in range(32)], [300, 200, 100, 50], 2304, "bf16")
    p = Plan(*args)
    assert p.geometry["mfma_path"] == 1 and p.geometry["two_pass"] == 1
    assert p.geometry["head_slices"] == 2
    # value rank 4096, 32 heads, 4 queries a sequence: eight slices of 16 rows
    # on the single-pass kernel; the two-pass kernels take the 128 rows too
    p4 = Plan(4096, 32, 32, 128, [i // 8 for i in range(32)], [300, 200, 100, 50], 4096, "bf16",
              queries_per_seq=4)
    assert p4.geometry["mfma_path"] == 1 and p4.geometry["two_pass"] == 1
    assert p4.geometry["head_slices"] == 8
    # an explicit single-pass plan, and two-pass requests the layer cannot
    # take: 512 (query, head) rows, fp32 latents
    assert Plan(*args, decode_passes=1).geometry["two_pass"] == 0
    assert Plan(*args, queries_per_seq=8, decode_passes=2).geometry["two_pass"] == 1
    from paper_2607_24331_amd import DckvError
    with pytest.raises(DckvError, match="decode_passes"):
        Plan(*args, queries_per_seq=16, decode_passes=2)
    with pytest.raises(DckvError, match="decode_passes"):
        Plan(*args[:-1], "f32", decode_passes=2)
    # explicit head slices
    wl = make_workload("mha_long_t128k")
    from paper_2607_24331_amd import Plan as P2
    p2 = P2(wl.hidden, 32, 32, 128, wl.group_of_kv, wl.group_rank, wl.value_rank, "bf16", 0, 2)
    assert p2.geometry["mfma_path"] == 1 and p2.geometry["head_slices"] == 2


def test_launch_info_reports_the_path():
    from paper_2607_24331_amd import Plan
    wl = make_workload("mha_long_t128k")
    args = (wl.hidden, 32, 32, 128, wl.group_of_kv, wl.group_rank, wl.value_rank, "bf16", 0)
    # one query: the single-pass split kernel, one slice
    i1 = Plan(*args).launch_info(1, 131072)
    assert i1["kernels"] == 1 and i1["head_slices"] == 1
    # four queries over 2048 pages: the two-pass kernels read the value part
    # once for the four slices; chunks of at most 64 pages
    p4 = Plan(*args, queries_per_seq=4)
    i4 = p4.launch_info(1, 131072)
    assert i4["kernels"] == 2 and i4["head_slices"] == 4
    assert 0 < i4["split_tokens"] <= 64 * 64 and i4["n_split"] * i4["split_tokens"] >= 131072
    # a short context stays on the single-pass kernel
    assert p4.launch_info(1, 4096)["kernels"] == 1
    assert Plan(*args, queries_per_seq=4, decode_passes=1).launch_info(1, 131072)["kernels"] == 1
    # many sequences of long context: the chunk search starts at the fewest
    # chunks the chunk-length cap allows, even past two work-groups a unit
    for q in (1, 4):
        p = Plan(*args, queries_per_seq=q, decode_passes=2)
        for batch in (64, 256):
            info = p.launch_info(batch, 131072)
            assert info["kernels"] == 2 and info["split_tokens"] > 0, (q, batch, info)
            assert info["n_split"] * info["split_tokens"] >= 131072
            assert p.workspace_bytes(batch, 131072) > 0


def test_queries_per_seq_plan():
    from paper_2607_24331_amd import Plan
    wl = make_workload("mha_long_t128k")
    args = (wl.hidden, 32, 32, 128, wl.group_of_kv, wl.group_rank, wl.value_rank, "bf16", 0)
    one = Plan(*args)
    assert one.geometry["queries_per_seq"] == 1 and one.geometry["head_slices"] == 1
    # 32 heads x 4 queries = 128 rows: four slices of 32 on the MFMA path
    four = Plan(*args, queries_per_seq=4)
    assert four.geometry["queries_per_seq"] == 4
    assert four.geometry["mfma_path"] == 1 and four.geometry["head_slices"] == 4
    # more workspace: one merged row per (sequence, query, head)
    assert four.workspace_bytes(1, 131072) > one.workspace_bytes(1, 131072)
    # 32 heads x 16 queries = 512 rows exceed the eight slices: portable path
    assert Plan(*args, queries_per_seq=16).geometry["mfma_path"] == 0


def test_group_order_cuts_the_smallest_group():
    from paper_2607_24331_amd import Plan
    # 32 query heads over 8 KV heads (4 each); groups of 2, 3 and 3 KV heads
    # (8, 12 and 12 rows) with ranks 96, 128, 160: key chunks 0-2, 3-6, 7-11.
    # Two 16-row tiles must cut one group; in group-id order that is group 1
    # (tiles load chunks 0-6 and 3-11: 16 loads), while cutting group 0
    # (tiles {g1 + 4 rows of g0}, {4 rows of g0 + g2}) loads 7 + 8 = 15.
    p = Plan(512, 32, 8, 64, [0, 0, 1, 1, 1, 2, 2, 2], [96, 128, 160], 256, "bf16")
    assert p.geometry["mfma_path"] == 1 and p.geometry["key_chunk_loads"] == 15
    # every group whole in one tile: each chunk loaded once
    p = Plan(512, 32, 8, 64, [0, 0, 0, 0, 1, 1, 1, 1], [96, 128], 256, "bf16")
    assert p.geometry["key_chunk_loads"] == 7
    # the GQA decode workload: groups of 8, 12 and 12 rows with 6, 8 and 10
    # chunks; cutting the 6-chunk group loads 30 chunks, and with 16 and 14
    # chunks a tile the 16-deep ring pads no key item
    g = _plan(make_workload("gqa8b_b4_t32k")).geometry
    assert g["key_chunk_loads"] == 30 and g["decode_ring"] == 16
    # the portable path reports none
    assert _plan(make_workload("tiny_mha_f32")).geometry["key_chunk_loads"] == 0


@pytest.mark.skipif(torch.cuda.is_available(), reason="raw fake pointers are only passed on a host without a GPU")
def test_rope_call_validation_never_launches(lib):
    from paper_2607_24331_amd import Plan
    A = 1 << 20
    n = ctypes.c_size_t()
    # the rotary decode runs on the bf16 MFMA path only, one query a sequence
    p32 = _plan(make_workload("tiny_mha_f32"))
    assert lib.dckv_rope_workspace_bytes(p32.handle, 1, 256, ctypes.byref(n)) == capi.DCKV_EINVAL
    assert "MFMA" in lib.dckv_last_error().decode()
    wl = make_workload("gqa8b_b4_t32k")
    pq = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
              wl.group_rank, wl.value_rank, wl.dtype, 0, queries_per_seq=4)
    assert lib.dckv_rope_workspace_bytes(pq.handle, 1, 256, ctypes.byref(n)) == capi.DCKV_EINVAL
    p = _plan(wl)
    assert lib.dckv_rope_workspace_bytes(p.handle, 4, 32768, ctypes.byref(n)) == capi.DCKV_OK
    need = n.value
    assert need > 0
    assert lib.dckv_rope_workspace_bytes(p.handle, 1, 1024, ctypes.byref(n)) == capi.DCKV_OK
    assert 0 < n.value < need
    args = [p.handle, A, 4, A, 4, A, 512, A, 32768, A, A, 10000.0, A, A, need, None]

    def call(**kw):
        a = list(args)
        idx = {"q": 1, "batch": 2, "num_pages": 4, "max_pages": 6, "max_context": 8,
               "base": 11, "out": 12, "ws": 13, "ws_bytes": 14}
        for k, v in kw.items():
            a[idx[k]] = v
        return lib.dckv_decode_rope(*a)
    for bad in (1.0, 0.5, float("nan"), float("inf"), -3.0):
        assert call(base=bad) == capi.DCKV_EINVAL
    assert call(q=None) == capi.DCKV_EINVAL
    assert call(max_context=512 * 64 + 1) == capi.DCKV_EINVAL
    assert call(out=A + 4) == capi.DCKV_EALIGN
    assert call(ws=A + 16) == capi.DCKV_EALIGN
    assert call(ws_bytes=need - 1) == capi.DCKV_EWORKSPACE
    assert call(batch=0) == capi.DCKV_OK
    assert lib.dckv_decode_rope(None, *args[1:]) == capi.DCKV_EINVAL
