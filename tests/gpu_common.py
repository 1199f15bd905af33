"""Shared helpers of the GPU parity tests: move seeded inputs to the device,
build pools with the oracle's layout, run the library, compare with the
oracle."""

from __future__ import annotations

import numpy as np
import torch

from oracle import append as oappend
from oracle import attention as oattn
from oracle import layout as olayout
from oracle.bookkeeping import book_for
from workloads.inputs import Inputs

TOL_REL_ROW = 2e-2      # max over rows of |o - o_ref|_inf / |o_ref|_inf (bf16 latents)
TOL_REL_ROW_F32 = 1e-4  # fp32 latents, fp32 accumulation


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.cuda()


def plan_for(wl, split_tokens: int = 0):
    from paper_2607_24331_amd import Plan
    return Plan(wl.hidden, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group_of_kv,
                wl.group_rank, wl.value_rank, wl.dtype, split_tokens)


def oracle_pool(inp: Inputs, with_append: bool = True) -> np.ndarray:
    """float32 pool packed by the oracle's layout: pre-filled latents, then
    the oracle's own append of x at the end of sequence 0."""
    wl = inp.wl
    pool = olayout.new_pool(inp.num_pages, wl.key_rank_total, wl.value_rank, dtype=np.float32)
    for b in range(wl.batch):
        if wl.prefill_lens[b]:
            olayout.pack(pool, inp.page_table, b, 0, inp.Zk_prefill[b], inp.Zv_prefill[b])
    if with_append and wl.append_tokens:
        Zk, Zv = oappend.latents(inp.x, inp.L_keys, inp.L_value, wl.dtype)
        olayout.pack(pool, inp.page_table, 0, wl.prefill_lens[0], Zk.astype(np.float32),
                     Zv.astype(np.float32))
    return pool


def append_slots(inp: Inputs) -> np.ndarray:
    wl = inp.wl
    pos = wl.prefill_lens[0] + np.arange(wl.append_tokens)
    return (inp.page_table[0, pos // 64].astype(np.int64) * 64 + pos % 64)


def gpu_pool_with_append(inp: Inputs, plan):
    """Device pool: pre-filled latents packed by the oracle layout (inputs),
    then the appended tokens written by the library's latent_append."""
    from paper_2607_24331_amd import latent_append
    wl = inp.wl
    pool = dev(oracle_pool(inp, with_append=False), wl.dtype)
    if wl.append_tokens:
        latent_append(plan, dev(inp.x, wl.dtype), dev(inp.L_keys.T, wl.dtype),
                      dev(inp.L_value.T, wl.dtype), torch.from_numpy(append_slots(inp)).cuda(), pool)
    return pool


def run_decode(inp: Inputs, plan, pool: torch.Tensor, q: np.ndarray = None) -> np.ndarray:
    from paper_2607_24331_amd import decode
    wl = inp.wl
    out = decode(plan, torch.from_numpy(np.ascontiguousarray(inp.q if q is None else q)).cuda(), pool,
                 torch.from_numpy(inp.page_table).cuda(), torch.from_numpy(inp.seq_lens).cuda(),
                 int(max(wl.seq_lens)) if wl.batch else 0,
                 dev(inp.R_keys_flat, wl.dtype), dev(inp.R_value, wl.dtype))
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def seq_latents(inp: Inputs, b: int):
    """Key and value latents [T_b, .] of sequence b as the oracle sees them:
    the seeded pre-filled latents, then (sequence 0) the oracle's append."""
    wl = inp.wl
    Zk = inp.Zk_prefill[b]
    Zv = inp.Zv_prefill[b]
    if b == 0 and wl.append_tokens:
        Zka, Zva = oappend.latents(inp.x, inp.L_keys, inp.L_value, wl.dtype)
        Zk = np.concatenate([Zk, Zka.astype(np.float32)])
        Zv = np.concatenate([Zv, Zva.astype(np.float32)])
    return Zk, Zv


def oracle_rows(inp: Inputs, pairs, q: np.ndarray = None) -> dict:
    """Oracle outputs of (sequence, head) pairs, from the seeded latents."""
    bk = book_for(inp.wl)
    q = inp.q if q is None else q
    res = {}
    by_b = {}
    for b, h in pairs:
        by_b.setdefault(b, []).append(h)
    for b, heads in sorted(by_b.items()):
        Zk, Zv = seq_latents(inp, b)
        for h in heads:
            res[(b, h)] = oattn.decode_head(q[b, h], Zk, Zv, inp.R_blocks, inp.R_value, bk, h,
                                            chunk=8192)
    return res


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    den = np.max(np.abs(ref))
    num = np.max(np.abs(got - ref))
    if den == 0:
        return float(num)
    return float(num / den)


def sample_pairs(wl, n: int, seed: int = 0):
    g = np.random.default_rng(seed)
    pairs = {(0, 0), (wl.batch - 1, wl.num_q_heads - 1)}
    # one head of every group at least
    for grp in range(wl.num_groups):
        kvs = [kv for kv in range(wl.num_kv_heads) if wl.group_of_kv[kv] == grp]
        h = kvs[int(g.integers(len(kvs)))] * (wl.num_q_heads // wl.num_kv_heads)
        pairs.add((int(g.integers(wl.batch)), h))
    while len(pairs) < n:
        pairs.add((int(g.integers(wl.batch)), int(g.integers(wl.num_q_heads))))
    return sorted(pairs)
