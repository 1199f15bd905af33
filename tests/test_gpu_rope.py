"""GPU parity of the rotary decode (dckv_decode_rope) against the oracle's
rotary reading: keys rebuilt from their group latent and turned by their
position, the query turned by the newest position (planes (i, i + d_h/2),
angle pos * base^(-2i/d_h)).

Small cases compare every row (several page rounds and splits, ragged
tails, a one-token and an empty sequence, GQA, singleton groups, groups
that start inside a 32-column key chunk, two 16-head tiles, d_h 64 and 128,
bases from fast- to slow-turning); the full-size layers compare sampled
rows at their real length (angles up to 1.3e5 radians).  Tolerance: 2e-2
relative per row, as for the position-free decode (bf16 latents, fp32
accumulation)."""

import numpy as np
import pytest
import torch

from oracle import rope as orope
from oracle.bookkeeping import book_for
from workloads import make_workload
from workloads.inputs import make_inputs

from gpu_common import (TOL_REL_ROW, dev, gpu_pool_with_append, plan_for, row_rel_err,
                        sample_pairs, seq_latents)
from test_gpu_parity import _small_inputs

pytestmark = pytest.mark.gpu


def _rope_rows(inp, pairs, base):
    wl = inp.wl
    bk = book_for(wl)
    res = {}
    for b, h in pairs:
        Zk, Zv = seq_latents(inp, b)
        res[(b, h)] = orope.decode_head(inp.q[b, h], Zk, Zv, inp.R_blocks, inp.R_value, bk, h, base,
                                        chunk=8192)
    return res


def _run(inp, plan, pool, base, max_context=None):
    from paper_2607_24331_amd import decode_rope
    wl = inp.wl
    out = decode_rope(plan, torch.from_numpy(np.ascontiguousarray(inp.q)).cuda(), pool,
                      torch.from_numpy(inp.page_table).cuda(), torch.from_numpy(inp.seq_lens).cuda(),
                      int(max(wl.seq_lens)) if max_context is None else max_context,
                      dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype), rope_base=base)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


# (case, base): the position-free decode's small cases that take the MFMA path
# (valu_bf16: value rank 2304 over 32 heads, two row slices of 16 heads)
CASES = [("mha_odd", 10000.0), ("gqa_uneven", 10000.0), ("single_group", 100.0),
         ("singletons", 500000.0), ("mha32_two_tiles", 10000.0), ("gqa_reordered", 1000.0),
         ("valu_bf16", 10000.0)]


@pytest.mark.parametrize("name, base", CASES)
def test_rope_small_all_rows(name, base):
    wl, inp, split = _small_inputs(name)
    plan = plan_for(wl, split)
    print(f"[rope] {name} base {base} split {split} d_h {wl.head_dim}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    out = _run(inp, plan, pool, base)
    ref = _rope_rows(inp, [(b, h) for b in range(wl.batch) for h in range(wl.num_q_heads)], base)
    errs = []
    for (b, h), o in ref.items():
        if wl.seq_lens[b] == 0:
            assert np.all(out[b, h] == 0)
            continue
        errs.append(row_rel_err(out[b, h], o))
    print(f"[rope] {name}: max row rel err {max(errs):.3e} over {len(errs)} rows", flush=True)
    assert max(errs) <= TOL_REL_ROW


def _wide_inputs(head_dim=128):
    # a group wider than the resident-factor kernel holds (14 key chunks at
    # d_h = 128, 28 at 64), so the general (per-chunk staging) kernel runs:
    # rank 470 spans 15 chunks; at d_h 64, rank 900 over 15 heads spans 29
    from test_gpu_parity import _groups
    from workloads.configs import custom_workload
    if head_dim == 128:
        lens, kvh, sizes, ranks = (1500, 70, 640), 8, (5, 3), (470, 96)
    else:
        lens, kvh, sizes, ranks = (700, 65), 16, (15, 1), (900, 40)
    wl = custom_workload(name=f"wide_group_d{head_dim}", seed=321, hidden=1024,
                         num_q_heads=2 * kvh, num_kv_heads=kvh, head_dim=head_dim,
                         group_of_kv=_groups(sizes, 11), group_rank=ranks, value_rank=256,
                         dtype="bf16", batch=len(lens), seq_lens=lens, prefill_lens=lens,
                         factor_scheme="orthonormal", permute_pages=True)
    return wl, make_inputs(wl)


@pytest.mark.parametrize("split, head_dim", [(512, 128), (1024, 128), (256, 64)])
def test_rope_wide_group_general_kernel(split, head_dim):
    wl, inp = _wide_inputs(head_dim)
    plan = plan_for(wl, split)
    print(f"[rope] wide_group d_h {head_dim} split {split}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    out = _run(inp, plan, pool, 10000.0)
    ref = _rope_rows(inp, [(b, h) for b in range(wl.batch) for h in range(wl.num_q_heads)], 10000.0)
    errs = [row_rel_err(out[b, h], o) for (b, h), o in ref.items()]
    print(f"[rope] wide_group d_h {head_dim}/{split}: max row rel err {max(errs):.3e} over {len(errs)} rows",
          flush=True)
    assert max(errs) <= TOL_REL_ROW


def test_rope_differs_from_position_free_and_is_reproducible():
    from paper_2607_24331_amd import decode
    wl, inp, split = _small_inputs("gqa_uneven")
    plan = plan_for(wl, split)
    pool = gpu_pool_with_append(inp, plan)
    a = _run(inp, plan, pool, 10000.0)
    b = _run(inp, plan, pool, 10000.0)
    assert np.array_equal(a, b)                          # fixed-order sums throughout
    plain = decode(plan, torch.from_numpy(inp.q).cuda(), pool, torch.from_numpy(inp.page_table).cuda(),
                   torch.from_numpy(inp.seq_lens).cuda(), int(max(wl.seq_lens)),
                   dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype)).cpu().numpy()
    assert np.max(np.abs(a - plain)) > 1e-2 * np.max(np.abs(plain))


def test_rope_split_lengths_agree():
    # the same rows through 64-, 256- and 1024-token splits (the cap): the
    # splits' partial softmaxes merge to the same result within rounding
    wl, inp, _ = _small_inputs("singletons")
    outs = []
    for split in (64, 256, 1024):
        plan = plan_for(wl, split)
        pool = gpu_pool_with_append(inp, plan)
        outs.append(_run(inp, plan, pool, 10000.0))
    for o in outs[1:]:
        for b in range(wl.batch):
            for h in range(wl.num_q_heads):
                assert row_rel_err(o[b, h], outs[0][b, h]) <= 1e-2


@pytest.mark.parametrize("name, n_rows", [("gqa8b_b4_t32k", 6), ("mha_long_t128k", 4),
                                          ("mha7b_b8_t4k", 6), ("mha_ragged_b64", 12)])
def test_rope_full_size_sampled_rows(name, n_rows):
    wl = make_workload(name)
    inp = make_inputs(wl)
    plan = plan_for(wl)
    print(f"[rope-full] {name}", flush=True)
    pool = gpu_pool_with_append(inp, plan)
    out = _run(inp, plan, pool, 10000.0)
    pairs = sample_pairs(wl, n_rows, seed=3)
    ref = _rope_rows(inp, pairs, 10000.0)
    errs = [row_rel_err(out[b, h], ref[(b, h)]) for b, h in pairs]
    print(f"[rope-full] {name}: max row rel err {max(errs):.3e} over {len(errs)} rows", flush=True)
    assert max(errs) <= TOL_REL_ROW
    assert np.all(np.isfinite(out))


def test_rope_rejects_plans_off_its_path():
    from paper_2607_24331_amd import DckvError, Plan, decode_rope
    wl, inp, split = _small_inputs("mha_odd", "f32")    # fp32 latents: the portable kernels
    plan = plan_for(wl, split)
    assert plan.geometry["mfma_path"] == 0
    pool = plan.new_pool(4)
    with pytest.raises(DckvError, match="MFMA"):
        decode_rope(plan, torch.zeros(1, wl.num_q_heads, wl.head_dim).cuda(), pool,
                    torch.zeros(1, 4, dtype=torch.int32).cuda(), torch.ones(1, dtype=torch.int32).cuda(),
                    64, torch.zeros(plan.key_factor_elems, dtype=plan.torch_dtype).cuda(),
                    torch.zeros(wl.value_rank, wl.num_kv_heads * wl.head_dim, dtype=plan.torch_dtype).cuda())
