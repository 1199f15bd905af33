"""Paged latent-cache layout (a stated reading: the paper caches z = x L per
token, Sec. III-A, but fixes no memory layout).

A pool is an array of pages; a page holds 64 consecutive token positions of
one sequence.  With R_K the total key rank and r_v the value rank, a page of
page_elems = 64 * R_Kp + 64 * r_v elements holds

  key part    [64 slots][R_Kp] token-major: element (slot s, key column k)
              at s * R_Kp + k; columns R_K .. R_Kp-1 are zero padding;
              group g's latent is columns koff_g .. koff_g + r_g - 1
  value part  [r_v][64] rank-major: element (slot s, value column j)
              at 64 * R_Kp + j * 64 + s

with R_Kp = R_K rounded up to a multiple of 8.  Token position pos of
sequence b lives in physical page page_table[b][pos // 64], slot pos % 64.
Slots past a sequence's length hold zeros in a freshly packed pool.
"""

from __future__ import annotations

import numpy as np

PAGE_TOKENS = 64


def key_row_stride(key_rank_total: int) -> int:
    return -(-key_rank_total // 8) * 8


def page_elems(key_rank_total: int, value_rank: int) -> int:
    return PAGE_TOKENS * key_row_stride(key_rank_total) + PAGE_TOKENS * value_rank


def value_base(key_rank_total: int) -> int:
    return PAGE_TOKENS * key_row_stride(key_rank_total)


def key_offset(slot: int, k: int, key_rank_total: int) -> int:
    return slot * key_row_stride(key_rank_total) + k


def value_offset(slot: int, j: int, key_rank_total: int) -> int:
    return value_base(key_rank_total) + j * PAGE_TOKENS + slot


def new_pool(num_pages: int, key_rank_total: int, value_rank: int, dtype=np.float64) -> np.ndarray:
    return np.zeros((num_pages, page_elems(key_rank_total, value_rank)), dtype=dtype)


def _page_views(pool, page, R_K, r_v):
    RKp = key_row_stride(R_K)
    keys = pool[page, :PAGE_TOKENS * RKp].reshape(PAGE_TOKENS, RKp)
    vals = pool[page, PAGE_TOKENS * RKp:PAGE_TOKENS * RKp + PAGE_TOKENS * r_v].reshape(r_v, PAGE_TOKENS)
    return keys, vals


def pack(pool: np.ndarray, page_table: np.ndarray, b: int, start: int,
         Zk: np.ndarray, Zv: np.ndarray) -> None:
    """Store the latents of positions start .. start+T-1 of sequence b."""
    T, R_K = Zk.shape
    r_v = Zv.shape[1]
    assert Zv.shape[0] == T
    pos = start
    while pos < start + T:
        page = int(page_table[b, pos // PAGE_TOKENS])
        s0 = pos % PAGE_TOKENS
        s1 = min(PAGE_TOKENS, s0 + (start + T - pos))
        t0 = pos - start
        t1 = t0 + (s1 - s0)
        keys, vals = _page_views(pool, page, R_K, r_v)
        keys[s0:s1, :R_K] = Zk[t0:t1]
        vals[:, s0:s1] = Zv[t0:t1].T
        pos += s1 - s0


def unpack(pool: np.ndarray, page_table: np.ndarray, b: int, T: int,
           key_rank_total: int, value_rank: int):
    """Latents (Zk [T, R_K], Zv [T, r_v]) of positions 0 .. T-1 of sequence b."""
    Zk = np.zeros((T, key_rank_total), dtype=pool.dtype)
    Zv = np.zeros((T, value_rank), dtype=pool.dtype)
    for p in range(-(-T // PAGE_TOKENS)):
        page = int(page_table[b, p])
        s1 = min(PAGE_TOKENS, T - p * PAGE_TOKENS)
        keys, vals = _page_views(pool, page, key_rank_total, value_rank)
        Zk[p * PAGE_TOKENS:p * PAGE_TOKENS + s1] = keys[:s1, :key_rank_total]
        Zv[p * PAGE_TOKENS:p * PAGE_TOKENS + s1] = vals[:, :s1].T
    return Zk, Zv
