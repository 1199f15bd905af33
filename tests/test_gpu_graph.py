"""Append + decode captured in a HIP graph (through torch.cuda.CUDAGraph on
the capture stream) and replayed, for serving loops that cannot launch
eagerly: every replay, with eager work and synchronisations in between,
must equal the eager result bit for bit."""

import numpy as np
import pytest
import torch

from gpu_common import append_slots, dev, oracle_pool
from workloads.configs import custom_workload
from workloads.inputs import make_inputs

pytestmark = pytest.mark.gpu


def _setup(Q=1):
    from paper_2607_24331_amd import Plan
    wl = custom_workload(name="graph_case", seed=41, hidden=512, num_q_heads=16, num_kv_heads=4,
                         head_dim=128, group_of_kv=(0, 1, 1, 0), group_rank=(200, 77),
                         value_rank=256, dtype="bf16", batch=2, seq_lens=(1000, 777),
                         prefill_lens=(936, 777), append_tokens=64, factor_scheme="orthonormal")
    inp = make_inputs(wl)
    plan = Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, 256, queries_per_seq=Q)
    pool = dev(oracle_pool(inp, with_append=False), wl.dtype)
    qshape = (wl.batch, Q, wl.num_q_heads, wl.head_dim) if Q > 1 else (wl.batch, wl.num_q_heads, wl.head_dim)
    q = torch.from_numpy(np.random.default_rng(3).standard_normal(qshape).astype(np.float32)).cuda()
    t = dict(x=dev(inp.x, wl.dtype), Lk=dev(inp.L_keys.T, wl.dtype), Lv=dev(inp.L_value.T, wl.dtype),
             slot=torch.from_numpy(append_slots(inp)).cuda(), pool=pool, q=q,
             table=torch.from_numpy(inp.page_table).cuda(), lens=torch.from_numpy(inp.seq_lens).cuda(),
             Rk=dev(inp.R_keys_flat, wl.dtype), Rv=dev(inp.R_value, wl.dtype))
    out = torch.empty(qshape, dtype=torch.float32, device="cuda")
    ws = plan.new_workspace(wl.batch, max(wl.seq_lens))
    return wl, plan, t, out, ws


@pytest.mark.parametrize("Q", [1, 3])
def test_graph_replays_equal_eager(Q):
    from paper_2607_24331_amd import decode, latent_append
    wl, plan, t, out, ws = _setup(Q)
    max_ctx = max(wl.seq_lens)

    def step():
        latent_append(plan, t["x"], t["Lk"], t["Lv"], t["slot"], t["pool"])
        decode(plan, t["q"], t["pool"], t["table"], t["lens"], max_ctx, t["Rk"], t["Rv"], out=out,
               workspace=ws)

    step()
    torch.cuda.synchronize()
    eager = out.clone()
    pool_eager = t["pool"].clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):                  # warm the capture stream first
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        out.fill_(float("nan"))                 # eager work between replays
        scratch = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r} differs"
        assert torch.equal(t["pool"], pool_eager), f"replay {r} pool differs"
        del scratch


def test_rotary_graph_replays_equal_eager():
    # the rotary decode (factor transpose, key rebuild, value pass, merge,
    # up-projection) records no memset and allocates nothing either
    from paper_2607_24331_amd import decode_rope, latent_append
    wl, plan, t, out, _ = _setup(1)
    max_ctx = max(wl.seq_lens)
    ws = torch.empty(plan.rope_workspace_bytes(wl.batch, max_ctx), dtype=torch.uint8, device="cuda")

    def step():
        latent_append(plan, t["x"], t["Lk"], t["Lv"], t["slot"], t["pool"])
        decode_rope(plan, t["q"], t["pool"], t["table"], t["lens"], max_ctx, t["Rk"], t["Rv"],
                    rope_base=10000.0, out=out, workspace=ws)

    step()
    torch.cuda.synchronize()
    eager = out.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        out.fill_(float("nan"))
        ws.fill_(0xAB)                          # stale workspace contents must not matter
        scratch = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r} differs"
        del scratch
