"""GPU: the decode entry point that allocates nothing (dckv_decode_noalloc,
scratch in a fixed device array) against dckv_decode with a caller
workspace, on two calls in a row through the C ABI -- the second with a
smaller input, so it runs over the scratch contents the first left -- each
also checked against the oracle; and an oversized call rejected with nothing
enqueued."""

import numpy as np
import pytest
import torch

from gpu_common import TOL_REL_ROW, dev, oracle_rows, plan_for, row_rel_err
from oracle import layout as olayout
from workloads.configs import custom_workload
from workloads.inputs import make_inputs

pytestmark = pytest.mark.gpu

LAYER = dict(hidden=1024, num_q_heads=32, num_kv_heads=8, head_dim=128,
             group_of_kv=(0, 1, 1, 2, 0, 2, 1, 2), group_rank=(192, 256, 320), value_rank=768,
             dtype="bf16", factor_scheme="orthonormal")


def _case(seed, seq_lens):
    wl = custom_workload(name=f"noalloc_{seed}", seed=seed, batch=len(seq_lens),
                         seq_lens=tuple(seq_lens), **LAYER)
    inp = make_inputs(wl)
    pool = olayout.new_pool(inp.num_pages, wl.key_rank_total, wl.value_rank, dtype=np.float32)
    for b in range(wl.batch):
        olayout.pack(pool, inp.page_table, b, 0, inp.Zk_prefill[b], inp.Zv_prefill[b])
    args = (torch.from_numpy(inp.q).cuda(), dev(pool, wl.dtype), torch.from_numpy(inp.page_table).cuda(),
            torch.from_numpy(inp.seq_lens).cuda(), int(max(seq_lens)), dev(inp.R_keys_flat, wl.dtype),
            dev(inp.R_value, wl.dtype))
    return wl, inp, args


def test_noalloc_matches_decode_on_two_calls():
    from paper_2607_24331_amd import decode, decode_noalloc
    from paper_2607_24331_amd.capi import NOALLOC_SCRATCH_BYTES
    first = _case(31, (8192, 5000, 7000, 3001))
    second = _case(32, (700, 65))                    # smaller: fewer sequences, shorter contexts
    plan = plan_for(first[0])
    assert plan.geometry["mfma_path"] == 1
    for wl, inp, args in (first, second):
        need = plan.workspace_bytes(wl.batch, args[4])
        assert 0 < need <= NOALLOC_SCRATCH_BYTES
        print(f"[noalloc] {wl.name} batch {wl.batch} max_context {args[4]} scratch {need} B",
              flush=True)
        ref = decode(plan, *args)
        out = torch.full_like(ref, float("nan"))
        got = decode_noalloc(plan, *args, out=out)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr()
        assert torch.equal(got, ref)                 # same kernels, same splits: bit for bit
        # and the oracle's bar on every row of the small call, sampled rows of the large one
        g = got.cpu().numpy().astype(np.float64)
        pairs = ([(b, h) for b in range(wl.batch) for h in range(wl.num_q_heads)] if wl.batch <= 2
                 else [(b, h) for b in range(wl.batch) for h in (0, 13, 31)])
        refs = oracle_rows(inp, pairs)
        err = max(row_rel_err(g[b, h], refs[(b, h)]) for b, h in pairs)
        print(f"[noalloc] {wl.name}: max row rel err {err:.2e} over {len(pairs)} rows", flush=True)
        assert err <= TOL_REL_ROW


def test_noalloc_rejects_oversized_call():
    from paper_2607_24331_amd import DckvError, decode_noalloc
    from paper_2607_24331_amd.capi import NOALLOC_SCRATCH_BYTES
    wl, inp, args = _case(33, (128,))
    q, pool, table, lens, ctx, rk, rv = args
    # 64-token splits over a declared bound of 131072 tokens: 2048 splits of
    # partials, beyond the array -- rejected on the host, nothing launched
    plan = plan_for(wl, split_tokens=64)
    big_ctx = 131072
    assert plan.workspace_bytes(1, big_ctx) > NOALLOC_SCRATCH_BYTES
    big_table = torch.full((1, big_ctx // 64), -1, dtype=torch.int32, device="cuda")
    big_table[:, :table.shape[1]] = table
    out = torch.full((1, wl.num_q_heads, wl.head_dim), 7.0, device="cuda")
    with pytest.raises(DckvError, match="scratch"):
        decode_noalloc(plan, q, pool, big_table, lens, big_ctx, rk, rv, out=out)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)
    # the same plan with the sequence's real bound fits and matches decode()
    got = decode_noalloc(plan, q, pool, table, lens, ctx, rk, rv, out=out)
    from paper_2607_24331_amd import decode
    ref = decode(plan, q, pool, table, lens, ctx, rk, rv)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
