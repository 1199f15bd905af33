"""Decode attention over the compressed cache, the plain way (fp64).

Per query head h of sequence b with T_b cached tokens:
  kv = floor(h / (H_q / H_kv)), g = group of kv, j = position of kv in g
  K_h = Z_g R_g[:, j d_h:(j+1) d_h]          keys rebuilt from the group latent
                                            (Sec. III-A x W ~ z R; Sec. III-C)
  V_h = Z_v R_v[:, kv d_h:(kv+1) d_h]        values rebuilt from the shared
                                            value latent (Sec. III-A; III-D)
  s_t = K_h[t] . q_h / sqrt(d_h)
  p   = exp(s - max s) / sum exp(s - max s)  (two passes over the scores)
  o_h = sum_t p_t V_h[t]

Readings where the paper is silent: softmax scale 1/sqrt(d_h); no positional
transform of keys; no mask (the decode query sees all T_b cached tokens);
T_b = 0 gives a zero output.

Several queries per sequence (speculative verification, chunked prefill):
the Q new tokens already occupy the last Q cache positions, query i sits at
position T_b - Q + i and sees every position up to its own (a causal mask
inside the chunk); a query that sees no position gives a zero output.  Long sequences are handled in token chunks:
pass one rebuilds keys chunk by chunk to get every score, pass two rebuilds
values chunk by chunk for the weighted sum -- the same arithmetic, in less
memory.
"""

from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

from . import layout as _layout
from .bookkeeping import Book


def _group_block(R_keys, book: Book, g: int) -> np.ndarray:
    if isinstance(R_keys, (list, tuple)):
        return np.asarray(R_keys[g], dtype=np.float64)
    flat = np.asarray(R_keys).reshape(-1)
    blk = flat[book.roff[g]:book.roff[g + 1]]
    return blk.reshape(book.ranks[g], book.heads_per_group[g] * book.head_dim).astype(np.float64)


def key_up(R_keys, book: Book, h: int) -> np.ndarray:
    """R_g[:, j d_h:(j+1) d_h] for query head h: r_g x d_h."""
    kv = book.kv_of_q[h]
    g = book.group_of_kv[kv]
    j = book.pos_in_group[kv]
    d = book.head_dim
    return _group_block(R_keys, book, g)[:, j * d:(j + 1) * d]


def value_up(R_value, book: Book, h: int) -> np.ndarray:
    """R_v[:, kv d_h:(kv+1) d_h] for query head h: r_v x d_h."""
    kv = book.kv_of_q[h]
    d = book.head_dim
    return np.asarray(R_value, dtype=np.float64)[:, kv * d:(kv + 1) * d]


def group_latent(Zk: np.ndarray, book: Book, g: int) -> np.ndarray:
    return Zk[:, book.koff[g]:book.koff[g] + book.ranks[g]]


def rebuild(Zk, Zv, R_keys, R_value, book: Book, h: int) -> Tuple[np.ndarray, np.ndarray]:
    """Full K_h [T, d_h] and V_h [T, d_h] of query head h."""
    g = book.group_of_kv[book.kv_of_q[h]]
    K = np.asarray(group_latent(Zk, book, g), dtype=np.float64) @ key_up(R_keys, book, h)
    V = np.asarray(Zv, dtype=np.float64) @ value_up(R_value, book, h)
    return K, V


def attend(q_h: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Textbook softmax attention of one query vector, fp64."""
    q_h = np.asarray(q_h, dtype=np.float64)
    s = (K @ q_h) / math.sqrt(q_h.shape[0])
    p = np.exp(s - s.max())
    p /= p.sum()
    return p @ V


def decode_head(q_h, Zk, Zv, R_keys, R_value, book: Book, h: int,
                chunk: Optional[int] = None) -> np.ndarray:
    """Output of query head h over latents Zk [T, R_K], Zv [T, r_v]."""
    T = Zk.shape[0]
    d = book.head_dim
    if T == 0:
        return np.zeros(d)
    if chunk is None or chunk >= T:
        K, V = rebuild(Zk, Zv, R_keys, R_value, book, h)
        return attend(q_h, K, V)
    q_h = np.asarray(q_h, dtype=np.float64)
    g = book.group_of_kv[book.kv_of_q[h]]
    Rk = key_up(R_keys, book, h)
    Rv = value_up(R_value, book, h)
    s = np.empty(T)
    for t0 in range(0, T, chunk):                       # pass 1: scores
        K = np.asarray(group_latent(Zk[t0:t0 + chunk], book, g), dtype=np.float64) @ Rk
        s[t0:t0 + chunk] = (K @ q_h) / math.sqrt(d)
    p = np.exp(s - s.max())
    p /= p.sum()
    o = np.zeros(d)
    for t0 in range(0, T, chunk):                       # pass 2: weighted values
        V = np.asarray(Zv[t0:t0 + chunk], dtype=np.float64) @ Rv
        o += p[t0:t0 + chunk] @ V
    return o


def decode(q: np.ndarray, pool: np.ndarray, page_table: np.ndarray, seq_lens: Sequence[int],
           R_keys, R_value, book: Book, pairs: Optional[Iterable[Tuple[int, int]]] = None,
           chunk: Optional[int] = 16384) -> np.ndarray:
    """Decode outputs [B, H_q, d_h] (fp64) read through the paged pool.

    With `pairs`, only those (sequence, head) rows are computed; the other
    rows are left NaN."""
    B, Hq, d = q.shape
    out = np.full((B, Hq, d), np.nan) if pairs is not None else np.zeros((B, Hq, d))
    todo: List[Tuple[int, int]] = (list(pairs) if pairs is not None
                                   else [(b, h) for b in range(B) for h in range(Hq)])
    by_seq = {}
    for b, h in todo:
        by_seq.setdefault(b, []).append(h)
    for b, heads in sorted(by_seq.items()):
        T = int(seq_lens[b])
        Zk, Zv = _layout.unpack(pool, page_table, b, T, book.key_rank_total, book.value_rank)
        for h in heads:
            out[b, h] = decode_head(q[b, h], Zk, Zv, R_keys, R_value, book, h, chunk=chunk)
    return out


def visible_tokens(T: int, Q: int, i: int) -> int:
    """Cache positions query i of Q sees in a sequence of T cached tokens."""
    return max(0, min(T, T - Q + i + 1))


def decode_multi(q: np.ndarray, pool: np.ndarray, page_table: np.ndarray,
                 seq_lens: Sequence[int], R_keys, R_value, book: Book,
                 rows: Optional[Iterable[Tuple[int, int, int]]] = None,
                 chunk: Optional[int] = 16384) -> np.ndarray:
    """Outputs [B, Q, H_q, d_h] (fp64) of Q queries per sequence, q [B, Q, H_q, d_h].

    With `rows`, only those (sequence, query, head) rows are computed; the
    others are left NaN."""
    B, Q, Hq, d = q.shape
    out = np.full((B, Q, Hq, d), np.nan) if rows is not None else np.zeros((B, Q, Hq, d))
    todo = (list(rows) if rows is not None
            else [(b, i, h) for b in range(B) for i in range(Q) for h in range(Hq)])
    by_seq = {}
    for b, i, h in todo:
        by_seq.setdefault(b, []).append((i, h))
    for b, qh in sorted(by_seq.items()):
        T = int(seq_lens[b])
        Zk, Zv = _layout.unpack(pool, page_table, b, T, book.key_rank_total, book.value_rank)
        for i, h in qh:
            n = visible_tokens(T, Q, i)
            out[b, i, h] = decode_head(q[b, i, h], Zk[:n], Zv[:n], R_keys, R_value, book, h,
                                       chunk=chunk)
    return out
