"""The five decode-layer workloads, each fully determined by a seed.

Shapes follow the paper's setting (Sec. III-C: a key projection of width
n = h * d_h split column-wise into groups of heads with ranks r_i; Sec. III-D:
one value latent of rank r over the whole projection) at the sizes of two
model families the paper targets (MHA and GQA attention, Sec. IV-A), scaled to
7B/8B-class layers.  The paper publishes no decode workload, so every shape
below is a stated choice, not a quotation.

Conventions (also recorded in the design notes):
  * query head h reads KV head floor(h / (H_q / H_kv));
  * the heads of a group are taken in ascending KV-head order, and groups are
    numbered in the listed order of their sizes;
  * seeded ranks: weight w_g = h_g * u_g with u_g ~ U[0.5, 1.5]; largest
    remainder rounding of total * w_g / sum(w) with ties to the lower group
    id; a group whose share exceeds h_g * d_h is pinned there and the excess
    is redistributed over the others (water-filling);
  * every random tensor is drawn from PCG64(SeedSequence([seed, tensor_id])).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Tuple

import numpy as np

PAGE_TOKENS = 64

# Stable ids of the random streams (one stream per drawn quantity).
STREAM_IDS: Dict[str, int] = {
    "head_perm": 1,
    "rank_importance": 2,
    "composition": 3,
    "seq_lens": 4,
    "page_perm": 5,
    "x": 10,
    "q": 11,
    "L_keys": 12,
    "L_value": 13,
    "R_keys": 14,
    "R_value": 15,
    "Zk_prefill": 16,
    "Zv_prefill": 17,
}


def rng_for(seed: int, stream: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, STREAM_IDS[stream]])))


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    hidden: int                      # m
    num_q_heads: int                 # H_q
    num_kv_heads: int                # H_kv (the paper's h)
    head_dim: int                    # d_h
    group_of_kv: Tuple[int, ...]     # [H_kv] -> group id
    group_rank: Tuple[int, ...]      # [G] key rank r_g
    value_rank: int                  # r_v
    dtype: str                       # "f32" or "bf16": latents, x and factors
    batch: int
    seq_lens: Tuple[int, ...]        # decode context per sequence (after append)
    prefill_lens: Tuple[int, ...]    # tokens whose latents are drawn directly
    append_tokens: int               # tokens appended through the down-projection
    factor_scheme: str               # "gaussian" | "orthonormal"
    permute_pages: bool              # physical pages in seeded order
    description: str = ""
    extra: dict = field(default_factory=dict, compare=False)

    # ---- derived shape facts (plain sums, no method arithmetic) ----
    @property
    def num_groups(self) -> int:
        return len(self.group_rank)

    @property
    def key_rank_total(self) -> int:
        return int(sum(self.group_rank))

    @property
    def kv_dim(self) -> int:
        return self.num_kv_heads * self.head_dim

    @property
    def group_sizes(self) -> Tuple[int, ...]:
        sizes = [0] * self.num_groups
        for g in self.group_of_kv:
            sizes[g] += 1
        return tuple(sizes)

    @property
    def pages_per_seq(self) -> Tuple[int, ...]:
        return tuple(-(-t // PAGE_TOKENS) for t in self.seq_lens)

    @property
    def max_pages(self) -> int:
        return max(self.pages_per_seq)

    @property
    def total_pages(self) -> int:
        return int(sum(self.pages_per_seq))

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


def _seeded_ranks(sizes, total, head_dim, rng) -> Tuple[int, ...]:
    """Ranks proportional to size x seeded importance, summing to `total`."""
    sizes = np.asarray(sizes, dtype=np.int64)
    G = len(sizes)
    u = rng.uniform(0.5, 1.5, size=G)
    w = sizes * u
    caps = sizes * head_dim
    pinned: Dict[int, int] = {}
    free = list(range(G))
    budget = int(total)
    while True:
        wf = w[free]
        quota = budget * wf / wf.sum()
        over = [g for g, qv in zip(free, quota) if qv > caps[g]]
        if not over:
            break
        for g in over:
            pinned[g] = int(caps[g])
            budget -= int(caps[g])
            free.remove(g)
    base = np.floor(quota).astype(np.int64)
    rem = quota - base
    short = budget - int(base.sum())
    order = sorted(range(len(free)), key=lambda i: (-rem[i], free[i]))
    for i in order[:short]:
        base[i] += 1
    ranks = [0] * G
    for g, r in pinned.items():
        ranks[g] = r
    for i, g in enumerate(free):
        ranks[g] = int(base[i])
    assert sum(ranks) == total, (ranks, total)
    assert all(1 <= r <= c for r, c in zip(ranks, caps)), (ranks, caps)
    return tuple(ranks)


def _groups_from_sizes(sizes, num_heads, rng) -> Tuple[int, ...]:
    """Seeded head permutation cut, in listed order, into groups of `sizes`."""
    perm = rng.permutation(num_heads)
    group_of = [-1] * num_heads
    pos = 0
    for g, s in enumerate(sizes):
        for h in perm[pos:pos + s]:
            group_of[int(h)] = g
        pos += s
    assert pos == num_heads and min(group_of) >= 0
    return tuple(group_of)


def _tiny_mha_f32() -> Workload:
    return Workload(
        name="tiny_mha_f32", seed=1, hidden=512, num_q_heads=8, num_kv_heads=8,
        head_dim=64, group_of_kv=(0, 1, 0, 1, 0, 1, 0, 1), group_rank=(48, 80),
        value_rank=128, dtype="f32", batch=1, seq_lens=(256,), prefill_lens=(0,),
        append_tokens=256, factor_scheme="gaussian", permute_pages=False,
        description="tiny MHA layer, fp32: m 512, 8 heads x 64, 1 x 256 tokens, "
                    "groups {0,2,4,6},{1,3,5,7} ranks {48,80}, value rank 128")


def _mha7b_b8_t4k() -> Workload:
    seed = 2
    sizes = (2, 3, 4, 4, 5, 6, 4, 4)
    group_of = _groups_from_sizes(sizes, 32, rng_for(seed, "head_perm"))
    ranks = _seeded_ranks(sizes, 2048, 128, rng_for(seed, "rank_importance"))
    return Workload(
        name="mha7b_b8_t4k", seed=seed, hidden=4096, num_q_heads=32, num_kv_heads=32,
        head_dim=128, group_of_kv=group_of, group_rank=ranks, value_rank=2048,
        dtype="bf16", batch=8, seq_lens=(4096,) * 8, prefill_lens=(4096,) * 8,
        append_tokens=0, factor_scheme="orthonormal", permute_pages=False,
        description="MHA 7B-shape layer, bf16: m 4096, 32 heads x 128, 8 x 4096 tokens, "
                    "8 seeded groups, key ranks sum 2048, value rank 2048")


def _gqa8b_b4_t32k() -> Workload:
    seed = 3
    sizes = (2, 3, 3)
    group_of = _groups_from_sizes(sizes, 8, rng_for(seed, "head_perm"))
    return Workload(
        name="gqa8b_b4_t32k", seed=seed, hidden=4096, num_q_heads=32, num_kv_heads=8,
        head_dim=128, group_of_kv=group_of, group_rank=(192, 256, 320), value_rank=768,
        dtype="bf16", batch=4, seq_lens=(32768,) * 4, prefill_lens=(32768,) * 4,
        append_tokens=0, factor_scheme="orthonormal", permute_pages=False,
        description="GQA 8B-shape layer, bf16: m 4096, 32 query / 8 KV heads x 128, "
                    "4 x 32768 tokens, groups {2,3,3} ranks {192,256,320}, value rank 768")


def _mha_long_t128k() -> Workload:
    seed = 4
    sizes = (8, 6, 6, 5, 4, 3)
    group_of = _groups_from_sizes(sizes, 32, rng_for(seed, "head_perm"))
    ranks = _seeded_ranks(sizes, 1536, 128, rng_for(seed, "rank_importance"))
    return Workload(
        name="mha_long_t128k", seed=seed, hidden=4096, num_q_heads=32, num_kv_heads=32,
        head_dim=128, group_of_kv=group_of, group_rank=ranks, value_rank=2048,
        dtype="bf16", batch=1, seq_lens=(131072,), prefill_lens=(131072 - 512,),
        append_tokens=512, factor_scheme="orthonormal", permute_pages=False,
        description="long-context MHA layer, bf16: m 4096, 32 heads x 128, 1 x 131072 "
                    "tokens (last 512 appended), 6 groups, key ranks sum 1536, value rank 2048")


def _mha_ragged_b64() -> Workload:
    seed = 5
    comp_rng = rng_for(seed, "composition")
    cuts = np.sort(comp_rng.choice(np.arange(1, 32), size=9, replace=False))
    edges = np.concatenate([[0], cuts, [32]])
    sizes = tuple(int(v) for v in np.diff(edges))
    group_of = _groups_from_sizes(sizes, 32, rng_for(seed, "head_perm"))
    ranks = _seeded_ranks(sizes, 1228, 128, rng_for(seed, "rank_importance"))
    lens = tuple(int(v) for v in rng_for(seed, "seq_lens").integers(1024, 8192, size=64, endpoint=True))
    return Workload(
        name="mha_ragged_b64", seed=seed, hidden=4096, num_q_heads=32, num_kv_heads=32,
        head_dim=128, group_of_kv=group_of, group_rank=ranks, value_rank=1536,
        dtype="bf16", batch=64, seq_lens=lens, prefill_lens=lens, append_tokens=0,
        factor_scheme="orthonormal", permute_pages=True,
        description="ragged paged MHA layer, bf16: m 4096, 32 heads x 128, 64 sequences "
                    "of U[1024,8192] tokens, 10 seeded groups, key ranks sum 1228, value rank 1536")


_BUILDERS = {
    "tiny_mha_f32": _tiny_mha_f32,
    "mha7b_b8_t4k": _mha7b_b8_t4k,
    "gqa8b_b4_t32k": _gqa8b_b4_t32k,
    "mha_long_t128k": _mha_long_t128k,
    "mha_ragged_b64": _mha_ragged_b64,
}

WORKLOAD_NAMES = tuple(_BUILDERS)


def make_workload(name: str) -> Workload:
    return _BUILDERS[name]()


def custom_workload(**kw) -> Workload:
    """A workload with explicit fields (unit tests and small parity cases)."""
    defaults = dict(name="custom", seed=0, factor_scheme="gaussian", permute_pages=False,
                    append_tokens=0, description="")
    defaults.update(kw)
    if "prefill_lens" not in defaults:
        defaults["prefill_lens"] = tuple(t - (defaults["append_tokens"] if i == 0 else 0)
                                         for i, t in enumerate(defaults["seq_lens"]))
    return Workload(**defaults)
