"""GPU parity of the two-pass decode kernels (score pass writing each page's
softmax weights with an integer exponent, value pass over value-rank groups,
chunk merge, up-projection) against the CPU oracle, on every output row of
small layers spanning ragged tails, empty and one-token sequences, singleton
groups, odd ranks, GQA, permuted pages, value ranks above 2048, and softmax
weights spread over hundreds of binary orders of magnitude."""

import numpy as np
import pytest
import torch

from gpu_common import TOL_REL_ROW, dev, gpu_pool_with_append, oracle_rows, row_rel_err, run_decode
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
