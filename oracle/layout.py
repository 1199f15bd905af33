"""Paged latent-cache layout (a stated reading: the paper caches z = x L per
token, Sec. III-A, but fixes no memory layout).

A pool is an array of pages; a page holds 64 consecutive token positions of
one sequence.  With R_K the total key rank and r_v the value rank, let
R_Kp = R_K rounded up to a multiple of 32 and r_vp = r_v rounded up to a
multiple of 16.  A page of page_elems = 64 * R_Kp + 64 * r_vp elements holds

  key part    chunk-major: key columns in chunks of 32; chunk c holds the 64
              slots one after another, 32 columns each.  Element (slot s,
              key column k) sits at (k // 32) * 2048 + s * 32 + k % 32.
              Columns R_K .. R_Kp-1 are zero padding.  Group g's latent is
              columns koff_g .. koff_g + r_g - 1.
  value part  tile-major, starting at 64 * R_Kp: value columns in tiles of
              16; tile u holds the slot halves 0-31 and 32-63 in turn, each
              as 16 columns x 32 slots.  Element (slot s, value column j)
              sits at 64 * R_Kp + (j // 16) * 1024 + (s // 32) * 512
              + (j % 16) * 32 + s % 32.  Columns r_v .. r_vp-1 are padding.

Token position pos of sequence b lives in physical page page_table[b][pos // 64],
slot pos % 64.  Slots past a sequence's length hold zeros in a freshly packed
pool.
"""

from __future__ import annotations

import numpy as np

PAGE_TOKENS = 64
KEY_CHUNK = 32
VALUE_TILE = 16


def key_width_padded(key_rank_total: int) -> int:
    return -(-key_rank_total // KEY_CHUNK) * KEY_CHUNK


def value_width_padded(value_rank: int) -> int:
    return -(-value_rank // VALUE_TILE) * VALUE_TILE


def page_elems(key_rank_total: int, value_rank: int) -> int:
    return PAGE_TOKENS * key_width_padded(key_rank_total) + PAGE_TOKENS * value_width_padded(value_rank)


def value_base(key_rank_total: int) -> int:
    return PAGE_TOKENS * key_width_padded(key_rank_total)


def key_offset(slot, k, key_rank_total: int):
    return (k // KEY_CHUNK) * (PAGE_TOKENS * KEY_CHUNK) + slot * KEY_CHUNK + k % KEY_CHUNK


def value_offset(slot, j, key_rank_total: int):
    half = PAGE_TOKENS // 2
    return (value_base(key_rank_total) + (j // VALUE_TILE) * (VALUE_TILE * PAGE_TOKENS)
            + (slot // half) * (VALUE_TILE * half) + (j % VALUE_TILE) * half + slot % half)


def new_pool(num_pages: int, key_rank_total: int, value_rank: int, dtype=np.float64) -> np.ndarray:
    return np.zeros((num_pages, page_elems(key_rank_total, value_rank)), dtype=dtype)


def _key_view(pool, page, R_K):
    """View of one page's key part: [chunks][64][32]."""
    RKp = key_width_padded(R_K)
    return pool[page, :PAGE_TOKENS * RKp].reshape(RKp // KEY_CHUNK, PAGE_TOKENS, KEY_CHUNK)


def _chunked(Z: np.ndarray, RKp: int) -> np.ndarray:
    """[T, R_K] -> [chunks][T][32], zero-padded to R_Kp columns."""
    T, R_K = Z.shape
    full = np.zeros((T, RKp), dtype=Z.dtype)
    full[:, :R_K] = Z
    return full.reshape(T, RKp // KEY_CHUNK, KEY_CHUNK).transpose(1, 0, 2)


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
        keys = _key_view(pool, page, R_K)
        keys[:, s0:s1, :] = _chunked(Zk[t0:t1], keys.shape[0] * KEY_CHUNK)
        slots = np.arange(s0, s1)[:, None]
        pool[page, value_offset(slots, np.arange(r_v)[None, :], R_K)] = Zv[t0:t1]
        pos += s1 - s0


def unpack(pool: np.ndarray, page_table: np.ndarray, b: int, T: int,
           key_rank_total: int, value_rank: int):
    """Latents (Zk [T, R_K], Zv [T, r_v]) of positions 0 .. T-1 of sequence b."""
    Zk = np.zeros((T, key_rank_total), dtype=pool.dtype)
    Zv = np.zeros((T, value_rank), dtype=pool.dtype)
    for p in range(-(-T // PAGE_TOKENS)):
        page = int(page_table[b, p])
        s1 = min(PAGE_TOKENS, T - p * PAGE_TOKENS)
        keys = _key_view(pool, page, key_rank_total)
        rows = keys[:, :s1, :].transpose(1, 0, 2).reshape(s1, -1)
        Zk[p * PAGE_TOKENS:p * PAGE_TOKENS + s1] = rows[:, :key_rank_total]
        slots = np.arange(s1)[:, None]
        Zv[p * PAGE_TOKENS:p * PAGE_TOKENS + s1] = pool[page, value_offset(
            slots, np.arange(value_rank)[None, :], key_rank_total)]
    return Zk, Zv
