"""Decode attention with rotary position embedding over the compressed cache
(fp64).  TEST INFRASTRUCTURE ONLY, like the rest of this package.

The paper never mentions positional encodings; this module states one
reading so that a position-aware decode has something to be checked against.

Rotation (RoFormer's rotary embedding, "rotate-half" pairing): with d = d_h,
coordinate i and coordinate i + d/2 (i < d/2) of a head vector span one
plane, turned by the angle pos * theta_i, theta_i = base^(-2i/d):
    x'_i       = x_i cos(pos theta_i) - x_{i+d/2} sin(pos theta_i)
    x'_{i+d/2} = x_{i+d/2} cos(pos theta_i) + x_i sin(pos theta_i)

Where it applies: the cache holds the latent of the key before rotation (the
factorisation of Sec. III-C is of the key projection, which precedes the
position transform), so the key of cache position t for query head h is
    K_h[t] = Rot(t) (Z_g[t] R_{g,h})          (keys rebuilt, then rotated)
and the decode query, the newest token at position T_b - 1, is rotated by
Rot(T_b - 1).  Values are not rotated.  Scores, softmax and the weighted sum
are those of the plain decode: s_t = K_h[t] . q'_h / sqrt(d_h), two passes.

`pos0` shifts every position (keys and query) by a constant; the method fixes
it at 0, and the tests use it to check that only position differences matter.
"""

from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

from . import layout as _layout
from .attention import group_latent, key_up, value_up
from .bookkeeping import Book


def frequencies(d: int, base: float) -> np.ndarray:
    """theta_i = base^(-2i/d), i = 0 .. d/2 - 1."""
    if d % 2:
        raise ValueError("the head dimension must be even")
    return float(base) ** (-2.0 * np.arange(d // 2) / d)


def rotate(X: np.ndarray, pos, base: float) -> np.ndarray:
    """Rot(pos) applied to the last axis of X [..., d]; pos broadcasts against
    X[..., 0] (one position per vector)."""
    X = np.asarray(X, dtype=np.float64)
    d = X.shape[-1]
    half = d // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * frequencies(d, base)
    c, s = np.cos(ang), np.sin(ang)
    a, b = X[..., :half], X[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def decode_head(q_h, Zk, Zv, R_keys, R_value, book: Book, h: int, base: float,
                pos0: int = 0, chunk: Optional[int] = None) -> np.ndarray:
    """Output of query head h over the latents Zk [T, R_K], Zv [T, r_v] of
    one sequence, with the rotary reading above."""
    T = Zk.shape[0]
    d = book.head_dim
    if T == 0:
        return np.zeros(d)
    chunk = T if chunk is None else chunk
    g = book.group_of_kv[book.kv_of_q[h]]
    Rk = key_up(R_keys, book, h)
    Rv = value_up(R_value, book, h)
    qr = rotate(q_h, pos0 + T - 1, base)
    s = np.empty(T)
    for t0 in range(0, T, chunk):                       # pass 1: rotated keys, scores
        K = np.asarray(group_latent(Zk[t0:t0 + chunk], book, g), dtype=np.float64) @ Rk
        pos = pos0 + np.arange(t0, t0 + K.shape[0])
        s[t0:t0 + chunk] = (rotate(K, pos, base) @ qr) / math.sqrt(d)
    p = np.exp(s - s.max())
    p /= p.sum()
    o = np.zeros(d)
    for t0 in range(0, T, chunk):                       # pass 2: weighted values
        V = np.asarray(Zv[t0:t0 + chunk], dtype=np.float64) @ Rv
        o += p[t0:t0 + chunk] @ V
    return o


def decode(q: np.ndarray, pool: np.ndarray, page_table: np.ndarray, seq_lens: Sequence[int],
           R_keys, R_value, book: Book, base: float,
           pairs: Optional[Iterable[Tuple[int, int]]] = None, pos0: int = 0,
           chunk: Optional[int] = 16384) -> np.ndarray:
    """Outputs [B, H_q, d_h] (fp64) read through the paged pool, q [B, H_q, d_h]
    before rotation.  With `pairs`, only those (sequence, head) rows are
    computed; the others are left NaN."""
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
            out[b, h] = decode_head(q[b, h], Zk, Zv, R_keys, R_value, book, h, base,
                                    pos0=pos0, chunk=chunk)
    return out
