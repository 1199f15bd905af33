"""GPU parity of the two-pass decode kernels (score pass writing each page's
softmax weights with an integer exponent, value pass over value-rank groups,
chunk merge, up-projection) against the CPU oracle, on every output row of
small layers spanning ragged tails, empty and one-token sequences, singleton
groups, odd ranks, GQA, permuted pages, value ranks above 2048, several causal
queries a sequence (one to eight row slices), and softmax weights spread over
hundreds of binary orders of magnitude."""

import numpy as np
import pytest
import torch

from gpu_common import (TOL_REL_ROW, dev, gpu_pool_with_append, oracle_pool, oracle_rows, row_rel_err,
                        run_decode)
from oracle import attention as oattn
from oracle.bookkeeping import book_for
from test_gpu_parity import SMALL, _all_rows, _report, _small_inputs
from workloads.configs import custom_workload
from workloads.inputs import make_inputs

pytestmark = pytest.mark.gpu


def _plan(wl, split=0, passes=2):
    from paper_2607_24331_amd import Plan
    p = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv, wl.group_rank,
             wl.value_rank, wl.dtype, split, decode_passes=passes)
    assert p.geometry["two_pass"] == (1 if passes == 2 else 0)
    return p


def _check_all(wl, inp, out, name, q=None):
    ref = _all_rows(inp, q=q)
    errs = []
    for (b, h), o in ref.items():
        if wl.seq_lens[b] == 0:
            assert np.all(out[b, h] == 0)
            continue
        errs.append(row_rel_err(out[b, h], o))
    _report(name, errs)
    assert max(errs) <= TOL_REL_ROW


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("chunked", [False, True])
def test_two_pass_small_all_rows(name, chunked):
    # chunked: value chunks of the case's split size (several chunks a
    # sequence, several waves' pages a chunk); else the default chunking
    wl, inp, split = _small_inputs(name)
    plan = _plan(wl, split if chunked else 0)
    print(f"[two-pass] {name} split {split if chunked else 'auto'}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    _check_all(wl, inp, out, f"two-pass/{name}/{'chunked' if chunked else 'auto'}")


@pytest.mark.parametrize("scale", [16.0, 300.0])
def test_two_pass_peaked_softmax(scale):
    # logits scaled far up: per-page exponents hundreds apart, pages whose
    # weights vanish against the running exponent, exact power-of-two rescales
    wl, inp, split = _small_inputs("singletons")
    plan = _plan(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    q = inp.q * scale
    out = run_decode(inp, plan, pool, q=q)
    assert np.isfinite(out).all()
    _check_all(wl, inp, out, f"two-pass/peaked x{scale:g}", q=q)


def test_two_pass_shift_of_all_logits():
    # softmax is invariant under a common shift; a query making every score
    # very negative (about -1e4 in base 2) must still give the plain average
    wl, inp, split = _small_inputs("single_group")
    plan = _plan(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    q = -inp.q * 2000.0
    out = run_decode(inp, plan, pool, q=q)
    assert np.isfinite(out).all()
    _check_all(wl, inp, out, "two-pass/very negative logits", q=q)


def test_two_pass_determinism_and_chunk_invariance():
    wl, inp, _ = _small_inputs("singletons")
    outs = []
    for split in (64, 192, 1024, 0):
        plan = _plan(wl, split)
        pool = gpu_pool_with_append(inp, plan)
        a = run_decode(inp, plan, pool)
        b = run_decode(inp, plan, pool)
        assert np.array_equal(a, b)                       # bitwise repeatable
        outs.append(a)
    for o in outs[1:]:
        assert np.max(np.abs(o - outs[0])) <= 1e-3 * np.max(np.abs(outs[0]))


def test_two_pass_page_permutation_is_invisible():
    wl, inp, split = _small_inputs("mha_odd")
    plan = _plan(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    out = run_decode(inp, plan, pool)
    g = np.random.default_rng(3)
    perm = g.permutation(inp.num_pages)
    pool2 = torch.empty_like(pool)
    pool2[torch.from_numpy(perm).cuda()] = pool
    inp.page_table = perm[inp.page_table].astype(np.int32)
    out2 = run_decode(inp, plan, pool2)
    assert np.array_equal(out, out2)


def test_two_pass_out_of_range_pages_and_nan_padding():
    # an invalid page entry inside a sequence reads as an empty page; NaN in
    # the slots past a sequence's end never reaches the output
    wl, inp, split = _small_inputs("gqa_uneven")
    plan = _plan(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    T = wl.seq_lens[1]
    last = inp.page_table[1, (T - 1) // 64]
    from oracle import layout as olayout
    RK, rv = wl.key_rank_total, wl.value_rank
    pad_slots = np.arange(T % 64, 64)
    if len(pad_slots):
        kidx = np.concatenate([olayout.key_offset(s, np.arange(RK), RK) for s in pad_slots])
        vidx = np.concatenate([olayout.value_offset(s, np.arange(rv), RK) for s in pad_slots])
        idx = torch.from_numpy(np.concatenate([kidx, vidx]).astype(np.int64)).cuda()
        row = pool[int(last)].clone()
        row[idx] = float("nan")
        pool[int(last)] = row
    out = run_decode(inp, plan, pool)
    assert np.isfinite(out).all()
    _check_all(wl, inp, out, "two-pass/nan padding")
    inp.page_table = inp.page_table.copy()
    inp.page_table[1, 3] = inp.num_pages + 5
    out = run_decode(inp, plan, pool)
    assert np.isfinite(out).all()


@pytest.mark.parametrize("rv", [2304, 4096])
def test_two_pass_large_value_rank(rv):
    # value ranks the single-pass kernel holds only 16 rows a slice for
    wl = custom_workload(name=f"rv{rv}", seed=rv, hidden=4096, num_q_heads=32, num_kv_heads=32,
                         head_dim=128, group_of_kv=tuple(i // 8 for i in range(32)),
                         group_rank=(300, 200, 100, 50), value_rank=rv, dtype="bf16", batch=2,
                         seq_lens=(333, 700), prefill_lens=(333, 700), factor_scheme="orthonormal")
    inp = make_inputs(wl)
    for passes in (2, 0):
        plan = _plan(wl, 0, passes) if passes == 2 else _plan(wl, 0, 1)
        assert plan.geometry["mfma_path"] == 1
        pool = gpu_pool_with_append(inp, plan)
        out = run_decode(inp, plan, pool)
        _check_all(wl, inp, out, f"rv{rv}/{'two-pass' if passes == 2 else 'single-pass'}")


@pytest.mark.parametrize("rv, lens", [(250, (129,)), (2048, (70, 1, 300)), (333, (64, 65))])
def test_few_rows_up_projection(rv, lens):
    # one to three rows a KV head over 32 KV heads: the up-projection that
    # reads whole 128-byte pieces of R_v rows; value ranks that are not a
    # multiple of 4 (element-wise staging of the merged rows) or of 128
    wl = custom_workload(name=f"few{rv}", seed=rv + len(lens), hidden=4096, num_q_heads=32,
                         num_kv_heads=32, head_dim=128, group_of_kv=tuple(i // 8 for i in range(32)),
                         group_rank=(96, 64, 160, 32), value_rank=rv, dtype="bf16",
                         batch=len(lens), seq_lens=lens, prefill_lens=lens,
                         factor_scheme="orthonormal")
    inp = make_inputs(wl)
    for passes in (2, 0):
        plan = _plan(wl, 0, passes) if passes == 2 else _plan(wl, 0, 1)
        print(f"[two-pass] few rows rv {rv} lens {lens} passes {passes}", flush=True)
        pool = gpu_pool_with_append(inp, plan)
        out = run_decode(inp, plan, pool)
        _check_all(wl, inp, out, f"few-rows/rv{rv}/{'two-pass' if passes == 2 else 'single-pass'}")


# (case, Q): several causal queries a sequence on the two-pass kernels.  Up
# to 32 rows take one slice (the per-wave value pass); beyond, 2 to 8 slices
# of up to 32 rows each share one walk over the value latents (4, 6, 8, 10,
# 12, 14 and 16 row tiles, each its own kernel instance); mha_odd holds a
# one-token and an empty sequence.
MULTI_PASS = [("singletons", 3), ("gqa_uneven", 4), ("mha_odd", 8), ("mha32_two_tiles", 2),
              ("mha32_two_tiles", 3), ("gqa_reordered", 4), ("mha32_two_tiles", 5),
              ("mha32_two_tiles", 6), ("mha32_two_tiles", 7), ("mha32_two_tiles", 8)]


def _multi_plan(wl, Q, split=0, passes=2):
    from paper_2607_24331_amd import Plan
    p = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
             wl.group_rank, wl.value_rank, wl.dtype, split, queries_per_seq=Q, decode_passes=passes)
    assert p.geometry["two_pass"] == (1 if passes == 2 else 0)
    return p


def _multi_check(wl, inp, plan, Q, name, scale=1.0, seed=11):
    from paper_2607_24331_amd import decode
    pool = gpu_pool_with_append(inp, plan)
    qm = (np.random.default_rng(seed).standard_normal(
        (wl.batch, Q, wl.num_q_heads, wl.head_dim)) * scale).astype(np.float32)
    out = decode(plan, torch.from_numpy(qm).cuda(), pool, torch.from_numpy(inp.page_table).cuda(),
                 torch.from_numpy(inp.seq_lens).cuda(), int(max(wl.seq_lens)),
                 dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype))
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    assert np.isfinite(got).all()
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
    _report(name, errs)
    assert max(errs) <= TOL_REL_ROW
    return got


@pytest.mark.parametrize("name, Q", MULTI_PASS)
@pytest.mark.parametrize("chunked", [False, True])
def test_two_pass_multi_query_all_rows(name, Q, chunked):
    wl, inp, split = _small_inputs(name)
    plan = _multi_plan(wl, Q, split if chunked else 0)
    info = plan.launch_info(wl.batch, int(max(wl.seq_lens)))
    assert info["kernels"] == 2
    print(f"[two-pass] {name} Q {Q} split {split if chunked else 'auto'} {info}", flush=True)
    _multi_check(wl, inp, plan, Q, f"two-pass/{name}/Q{Q}/{'chunked' if chunked else 'auto'}")


@pytest.mark.parametrize("scale", [16.0, 300.0])
def test_two_pass_multi_query_peaked_softmax(scale):
    # per-page exponents far apart: the staged weights rescaled to running
    # exponents that change from page to page, the accumulators with them
    wl, inp, split = _small_inputs("gqa_reordered")
    plan = _multi_plan(wl, 4, 64)
    _multi_check(wl, inp, plan, 4, f"two-pass/Q4 peaked x{scale:g}", scale=scale)


def test_two_pass_multi_query_matches_single_pass_bitwise_stable():
    # both kernel sets on the same rows, each bitwise repeatable
    wl, inp, split = _small_inputs("mha32_two_tiles")
    a = _multi_check(wl, inp, _multi_plan(wl, 4, 0), 4, "two-pass/Q4")
    b = _multi_check(wl, inp, _multi_plan(wl, 4, 0), 4, "two-pass/Q4 again")
    assert np.array_equal(a, b)
    c = _multi_check(wl, inp, _multi_plan(wl, 4, 256, passes=1), 4, "single-pass/Q4")
    assert np.max(np.abs(a - c)) <= 2e-2 * np.max(np.abs(c))


def test_two_pass_multi_query_wide_value_groups():
    # 64 rows (four row tiles) over enough pages that a value work-group
    # takes 16 tiles (two a wave) over chunks of several pages
    wl = custom_workload(name="q2_rv2048", seed=2048, hidden=4096, num_q_heads=32, num_kv_heads=32,
                         head_dim=128, group_of_kv=tuple(i // 8 for i in range(32)),
                         group_rank=(300, 200, 100, 50), value_rank=2048, dtype="bf16", batch=2,
                         seq_lens=(16384, 9001), prefill_lens=(16384, 9001),
                         factor_scheme="orthonormal")
    inp = make_inputs(wl)
    plan = _multi_plan(wl, 2)
    info = plan.launch_info(wl.batch, 16384)
    assert info["kernels"] == 2 and info["head_slices"] == 2 and info["value_tiles"] == 16, info
    print(f"[two-pass] q2_rv2048 {info}", flush=True)
    _multi_check(wl, inp, plan, 2, "two-pass/q2_rv2048")
