"""Uncompressed KV decode, the plain way (fp64) -- the baseline the compressed
cache is measured against (test infrastructure only, like the rest of this
package: nothing in the product path imports it).

Each query head h of sequence b attends to the T_b cached keys and values of
its KV head kv = floor(h / (H_q / H_kv)) (the same head map as the compressed
path), with softmax scale 1/sqrt(d_h) and no mask:
  o_h = softmax(K_kv q_h / sqrt(d_h)) V_kv

Paged layout of the uncompressed cache (a stated reading, like the latent
layout: 64 tokens a page):
  key part    [H_kv][64][d_h]: (slot s, KV head kv, column d) at (kv*64 + s)*d_h + d
  value part  the same, after the 64*H_kv*d_h key elements
so one head's keys of a page are one contiguous run of 64*d_h elements.
"""

from __future__ import annotations

from typing import Sequence

import numpy as np

from .attention import attend

PAGE_TOKENS = 64


def page_elems(num_kv_heads: int, head_dim: int) -> int:
    return 2 * PAGE_TOKENS * num_kv_heads * head_dim


def key_offset(slot, kv, d, num_kv_heads: int, head_dim: int):
    return (kv * PAGE_TOKENS + slot) * head_dim + d


def value_offset(slot, kv, d, num_kv_heads: int, head_dim: int):
    return PAGE_TOKENS * num_kv_heads * head_dim + (kv * PAGE_TOKENS + slot) * head_dim + d


def new_pool(num_pages: int, num_kv_heads: int, head_dim: int, dtype=np.float64) -> np.ndarray:
    return np.zeros((num_pages, page_elems(num_kv_heads, head_dim)), dtype=dtype)


def pack(pool, page_table, b: int, start: int, K: np.ndarray, V: np.ndarray) -> None:
    """Store keys and values [T, H_kv, d_h] of positions start .. start+T-1."""
    T, Hkv, d = K.shape
    kv = np.arange(Hkv)[None, :, None]
    dd = np.arange(d)[None, None, :]
    for t in range(T):
        pos = start + t
        page = int(page_table[b, pos // PAGE_TOKENS])
        s = pos % PAGE_TOKENS
        pool[page, key_offset(s, kv, dd, Hkv, d)] = K[t][None]
        pool[page, value_offset(s, kv, dd, Hkv, d)] = V[t][None]


def unpack(pool, page_table, b: int, T: int, num_kv_heads: int, head_dim: int):
    """Keys and values [T, H_kv, d_h] of positions 0 .. T-1 of sequence b."""
    K = np.zeros((T, num_kv_heads, head_dim), dtype=pool.dtype)
    V = np.zeros_like(K)
    kv = np.arange(num_kv_heads)[:, None]
    dd = np.arange(head_dim)[None, :]
    for t in range(T):
        page = int(page_table[b, t // PAGE_TOKENS])
        s = t % PAGE_TOKENS
        K[t] = pool[page, key_offset(s, kv, dd, num_kv_heads, head_dim)]
        V[t] = pool[page, value_offset(s, kv, dd, num_kv_heads, head_dim)]
    return K, V


def decode(q: np.ndarray, pool: np.ndarray, page_table: np.ndarray, seq_lens: Sequence[int],
           num_kv_heads: int) -> np.ndarray:
    """Outputs [B, H_q, d_h] (fp64) of one query per sequence; T_b = 0 gives zeros."""
    B, Hq, d = q.shape
    qpk = Hq // num_kv_heads
    out = np.zeros((B, Hq, d))
    for b in range(B):
        T = int(seq_lens[b])
        if T == 0:
            continue
        K, V = unpack(pool, page_table, b, T, num_kv_heads, d)
        for h in range(Hq):
            kv = h // qpk
            out[b, h] = attend(q[b, h], K[:, kv].astype(np.float64), V[:, kv].astype(np.float64))
    return out
