"""Latent write for new tokens (Sec. III-A: the cache stores z = x L instead of
x W; Sec. III-C: the key latent of group i is x L_i; Sec. III-D: the value
latent is x L_v over the whole projection).

The exact product is formed in fp64 and rounded once to the storage type
(bf16 round-to-nearest-even, or fp32), then placed by the layout.
"""

from __future__ import annotations

import numpy as np

from . import bf16 as _bf16
from . import layout as _layout


def down_project(x: np.ndarray, L: np.ndarray) -> np.ndarray:
    """z = x L in fp64 (one row per token)."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(L, dtype=np.float64)


def latents(x, L_keys, L_value, dtype: str):
    """Rounded key latent [T, R_K] (groups side by side) and value latent [T, r_v]."""
    Zk = _bf16.round_storage(down_project(x, L_keys), dtype)
    Zv = _bf16.round_storage(down_project(x, L_value), dtype)
    return Zk, Zv


def append(pool: np.ndarray, page_table: np.ndarray, b: int, start: int,
           x, L_keys, L_value, dtype: str) -> None:
    """Write the latents of rows of x as positions start.. of sequence b."""
    Zk, Zv = latents(x, L_keys, L_value, dtype)
    _layout.pack(pool, page_table, b, start, Zk, Zv)


def abs_bound(x, L) -> np.ndarray:
    """sum_k |x_k| |L_kj| per output: scales the accumulation error of any
    summation order (used to state tolerances, not a result)."""
    return np.abs(np.asarray(x, dtype=np.float64)) @ np.abs(np.asarray(L, dtype=np.float64))
