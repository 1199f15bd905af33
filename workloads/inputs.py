"""Seeded input tensors for a Workload (host numpy arrays).

Everything here is input construction: random draws, rounding of the draws
to the storage dtype, QR orthonormalisation of random factor matrices and the
page table.  Values destined for bf16 storage are returned as float32 arrays
whose every element is exactly a bf16 value, so both sides read identical
numbers.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np
import torch

from .configs import PAGE_TOKENS, Workload, rng_for


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are exactly bf16 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("array holds values that are not exact bf16 values")
    return (u >> 16).astype(np.uint16)


def f32_from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """float32 values of uint16 bf16 bit patterns (exact widening)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round random float draws to the storage dtype, returned as float32."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a32
    return torch.from_numpy(a32).to(torch.bfloat16).to(torch.float32).numpy()


def _normal(seed: int, stream: str, shape, std: float = 1.0) -> np.ndarray:
    g = rng_for(seed, stream)
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def _orthonormal_rows(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    """rows x cols matrix with orthonormal rows (rows <= cols), float64."""
    g = rng.standard_normal(size=(cols, rows))
    q, r = np.linalg.qr(g, mode="reduced")
    q *= np.sign(np.diag(r))[None, :]
    return q.T.copy()


@dataclass
class Inputs:
    wl: Workload
    x: np.ndarray                 # [append_tokens, m] (storage-exact float32)
    q: np.ndarray                 # [B, H_q, d_h] float32
    L_keys: np.ndarray            # [m, R_K]  = [L_0 | ... | L_{G-1}]
    L_value: np.ndarray           # [m, r_v]
    R_blocks: List[np.ndarray]    # per group [r_g, h_g*d_h]
    R_value: np.ndarray           # [r_v, n]
    Zk_prefill: List[np.ndarray]  # per sequence [prefill_b, R_K]
    Zv_prefill: List[np.ndarray]  # per sequence [prefill_b, r_v]
    page_table: np.ndarray        # [B, max_pages] int32
    seq_lens: np.ndarray          # [B] int32
    num_pages: int                # physical pages in the pool

    @property
    def R_keys_flat(self) -> np.ndarray:
        """Concatenation of the row-major R_g blocks, group 0 first."""
        return np.concatenate([b.reshape(-1) for b in self.R_blocks]).astype(np.float32)


def make_page_table(wl: Workload) -> np.ndarray:
    pages = wl.pages_per_seq
    total = int(sum(pages))
    if wl.permute_pages:
        phys = rng_for(wl.seed, "page_perm").permutation(total).astype(np.int32)
    else:
        phys = np.arange(total, dtype=np.int32)
    table = np.zeros((wl.batch, wl.max_pages), dtype=np.int32)
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = phys[pos:pos + n]
        pos += n
    return table


def make_factors(wl: Workload):
    m, r_v, n = wl.hidden, wl.value_rank, wl.kv_dim
    RK = wl.key_rank_total
    dt = wl.dtype
    sizes = wl.group_sizes
    if wl.factor_scheme == "gaussian":
        L_keys = to_storage(_normal(wl.seed, "L_keys", (m, RK), 1.0 / np.sqrt(m)), dt)
        L_value = to_storage(_normal(wl.seed, "L_value", (m, r_v), 1.0 / np.sqrt(m)), dt)
        g = rng_for(wl.seed, "R_keys")
        R_blocks = [to_storage(g.standard_normal((r, h * wl.head_dim)) / np.sqrt(r), dt)
                    for r, h in zip(wl.group_rank, sizes)]
        R_value = to_storage(_normal(wl.seed, "R_value", (r_v, n), 1.0 / np.sqrt(r_v)), dt)
    elif wl.factor_scheme == "orthonormal":
        L_keys = to_storage(_normal(wl.seed, "L_keys", (m, RK), 1.0 / np.sqrt(m)), dt)
        L_value = to_storage(_normal(wl.seed, "L_value", (m, r_v), 1.0 / np.sqrt(m)), dt)
        g = rng_for(wl.seed, "R_keys")
        R_blocks = [to_storage(_orthonormal_rows(g, r, h * wl.head_dim), dt)
                    for r, h in zip(wl.group_rank, sizes)]
        R_value = to_storage(_orthonormal_rows(rng_for(wl.seed, "R_value"), r_v, n), dt)
    else:
        raise ValueError(wl.factor_scheme)
    return L_keys, L_value, R_blocks, R_value


def make_inputs(wl: Workload, with_prefill: bool = True, with_factors: bool = True) -> Inputs:
    m, r_v = wl.hidden, wl.value_rank
    RK = wl.key_rank_total
    dt = wl.dtype
    x = to_storage(_normal(wl.seed, "x", (wl.append_tokens, m)), dt)
    q = _normal(wl.seed, "q", (wl.batch, wl.num_q_heads, wl.head_dim))
    if with_factors:
        L_keys, L_value, R_blocks, R_value = make_factors(wl)
    else:
        L_keys = L_value = R_value = None
        R_blocks = []
    Zk, Zv = [], []
    if with_prefill:
        gk = rng_for(wl.seed, "Zk_prefill")
        gv = rng_for(wl.seed, "Zv_prefill")
        for t in wl.prefill_lens:
            Zk.append(to_storage(gk.standard_normal((t, RK), dtype=np.float32), dt))
            Zv.append(to_storage(gv.standard_normal((t, r_v), dtype=np.float32), dt))
    table = make_page_table(wl)
    return Inputs(wl=wl, x=x, q=q, L_keys=L_keys, L_value=L_value, R_blocks=R_blocks,
                  R_value=R_value, Zk_prefill=Zk, Zv_prefill=Zv, page_table=table,
                  seq_lens=np.asarray(wl.seq_lens, dtype=np.int32), num_pages=wl.total_pages)


def random_pool_fill(num_pages: int, page_elems: int, dtype: str, seed: int,
                     device: Optional[str] = None) -> torch.Tensor:
    """A pool of i.i.d. N(0,1) storage values drawn by torch (benchmark use).

    Every element, padding included, is a finite random value; a correct
    decode ignores the slots past each sequence's length.
    """
    gen = torch.Generator(device=device or "cpu")
    gen.manual_seed(seed)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    return torch.randn((num_pages, page_elems), generator=gen, device=device, dtype=torch.float32).to(tdt)


__all__ = ["Inputs", "make_inputs", "make_factors", "make_page_table", "bf16_bits_from_f32",
           "f32_from_bf16_bits", "to_storage", "random_pool_fill", "PAGE_TOKENS"]
