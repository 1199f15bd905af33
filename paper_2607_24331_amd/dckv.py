"""Python binding of libdckv (argument marshalling only).

Every step of append and decode runs in the HIP kernels behind the C ABI;
PyTorch supplies device memory and the current stream.  The functions take
torch tensors on the GPU, check their dtypes, shapes and contiguity against
the plan, and pass raw pointers down.
"""

from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from . import capi

_lib = capi.load()

_DTYPES = {"f32": (capi.DCKV_F32, torch.float32), "bf16": (capi.DCKV_BF16, torch.bfloat16)}


class DckvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib.dckv_last_error().decode(errors="replace")
        super().__init__(f"{where}: {capi.STATUS_NAMES.get(status, status)}: {msg}")


def _check(status: int, where: str) -> None:
    if status != capi.DCKV_OK:
        raise DckvError(status, where)


def _i32_array(values: Sequence[int]):
    arr = (ctypes.c_int32 * len(values))(*[int(v) for v in values])
    return arr


class Plan:
    """Host plan of one layer: grouping, ranks, layout and split size."""

    def __init__(self, hidden: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 group_of_kv_head: Sequence[int], group_rank: Sequence[int], value_rank: int,
                 dtype: str = "bf16", split_tokens: int = 0, head_slices: int = 0,
                 decode_waves: int = 0, queries_per_seq: int = 1, decode_passes: int = 0):
        if dtype not in _DTYPES:
            raise ValueError(f"dtype must be one of {sorted(_DTYPES)}")
        self.dtype = dtype
        self.torch_dtype = _DTYPES[dtype][1]
        self._gmap = _i32_array(group_of_kv_head)
        self._ranks = _i32_array(group_rank)
        desc = capi.LayerDesc(hidden, num_q_heads, num_kv_heads, head_dim, len(group_rank),
                              ctypes.cast(self._gmap, ctypes.POINTER(ctypes.c_int32)),
                              ctypes.cast(self._ranks, ctypes.POINTER(ctypes.c_int32)),
                              value_rank, _DTYPES[dtype][0], split_tokens, head_slices,
                              queries_per_seq, decode_waves, decode_passes)
        handle = ctypes.c_void_p()
        _check(_lib.dckv_plan_create(ctypes.byref(desc), ctypes.byref(handle)), "plan_create")
        self._handle = handle
        self.hidden, self.num_q_heads, self.num_kv_heads = hidden, num_q_heads, num_kv_heads
        self.head_dim, self.num_groups, self.value_rank = head_dim, len(group_rank), value_rank
        info = self.info()
        self.geometry = info["geometry"]
        self.key_rank_total = self.geometry["key_rank_total"]
        self.key_width_padded = self.geometry["key_width_padded"]
        self.page_elems = self.geometry["page_elems"]
        self.split_tokens = self.geometry["split_tokens"]
        self.key_factor_elems = self.geometry["key_factor_elems"]
        self.queries_per_seq = self.geometry["queries_per_seq"]

    @property
    def handle(self) -> ctypes.c_void_p:
        if self._handle is None:
            raise ValueError("plan is closed")
        return self._handle

    def info(self) -> dict:
        geo = capi.PlanGeometry()
        G, Hkv, Hq = self.num_groups, self.num_kv_heads, self.num_q_heads
        koff = (ctypes.c_int32 * G)()
        pos = (ctypes.c_int32 * Hkv)()
        qoff = (ctypes.c_int32 * (Hq + 1))()
        roff = (ctypes.c_int64 * (G + 1))()
        _check(_lib.dckv_plan_info(self.handle, ctypes.byref(geo), koff, pos, qoff, roff), "plan_info")
        return {
            "geometry": {name: getattr(geo, name) for name, _ in capi.PlanGeometry._fields_},
            "koff": list(koff), "pos_in_group": list(pos), "qoff": list(qoff), "roff": list(roff),
        }

    def workspace_bytes(self, batch: int, max_context: int) -> int:
        n = ctypes.c_size_t()
        _check(_lib.dckv_decode_workspace_bytes(self.handle, batch, max_context, ctypes.byref(n)),
               "decode_workspace_bytes")
        return n.value

    def launch_info(self, batch: int, max_context: int) -> dict:
        """The launch a decode of `batch` sequences of at most `max_context`
        tokens takes: kernels (0 portable, 1 single-pass, 2 two-pass),
        split_tokens, n_split, head_slices, value_tiles."""
        info = capi.LaunchInfo()
        _check(_lib.dckv_decode_launch_info(self.handle, batch, max_context, ctypes.byref(info)),
               "decode_launch_info")
        return {name: getattr(info, name) for name, _ in capi.LaunchInfo._fields_}

    def rope_workspace_bytes(self, batch: int, max_context: int) -> int:
        n = ctypes.c_size_t()
        _check(_lib.dckv_rope_workspace_bytes(self.handle, batch, max_context, ctypes.byref(n)),
               "rope_workspace_bytes")
        return n.value

    def new_pool(self, num_pages: int, device="cuda") -> torch.Tensor:
        """Zero-filled pool of `num_pages` pages."""
        return torch.zeros((num_pages, self.page_elems), dtype=self.torch_dtype, device=device)

    def new_workspace(self, batch: int, max_context: int, device="cuda") -> torch.Tensor:
        n = self.workspace_bytes(batch, max_context)
        return torch.empty(max(n, 256), dtype=torch.uint8, device=device)

    def set_profile_events(self, before=None, after=None) -> None:
        """Record two torch.cuda.Event objects around the split-K attention
        kernel of every later decode (benchmark instrumentation); None stops."""
        hb = before.cuda_event if before is not None else None
        ha = after.cuda_event if after is not None else None
        _check(_lib.dckv_plan_set_profile_events(self.handle, hb, ha), "plan_set_profile_events")

    def close(self) -> None:
        if getattr(self, "_handle", None) is not None:
            _lib.dckv_plan_destroy(self._handle)
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dev(t: torch.Tensor, name: str, dtype, shape=None) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


def _num_pages(plan: Plan, pool: torch.Tensor) -> int:
    if pool.numel() % plan.page_elems:
        raise ValueError("pool size is not a whole number of pages")
    return pool.numel() // plan.page_elems


def latent_append(plan: Plan, x: torch.Tensor, L_keys: torch.Tensor, L_value: torch.Tensor,
                  slot: torch.Tensor, pool: torch.Tensor, stream=None) -> None:
    """Write z = x L of each row of x into its pool slot.  L_keys [R_K, m] and
    L_value [r_v, m] hold the factors transposed ([out, in], as a linear
    layer's weight)."""
    n_tok = x.shape[0] if x.dim() == 2 else -1
    dt = plan.torch_dtype
    px = _dev(x, "x", dt, (n_tok, plan.hidden))
    pk = _dev(L_keys, "L_keys", dt, (plan.key_rank_total, plan.hidden))
    pv = _dev(L_value, "L_value", dt, (plan.value_rank, plan.hidden))
    ps = _dev(slot, "slot", torch.int64, (n_tok,))
    pp = _dev(pool, "pool", dt)
    _check(_lib.dckv_latent_append(plan.handle, px, n_tok, pk, pv, ps, pp, _num_pages(plan, pool),
                                   _stream_handle(stream)), "latent_append")


def decode(plan: Plan, q: torch.Tensor, pool: torch.Tensor, page_table: torch.Tensor,
           seq_lens: torch.Tensor, max_context: int, R_keys: torch.Tensor, R_value: torch.Tensor,
           out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
           stream=None) -> torch.Tensor:
    """Attention output (fp32) of the plan's Q queries per sequence: q and the
    result are [batch, Q, H_q, d_h], or [batch, H_q, d_h] when Q is 1.  Query
    i of sequence b sits at cache position seq_len - Q + i and sees every
    position up to its own."""
    Q = plan.queries_per_seq
    if q.dim() == 3 and Q == 1:
        qshape = (q.shape[0], plan.num_q_heads, plan.head_dim)
    elif q.dim() == 4:
        qshape = (q.shape[0], Q, plan.num_q_heads, plan.head_dim)
    else:
        raise ValueError("q must be [batch, Q, H_q, d_h] (or [batch, H_q, d_h] with Q = 1)")
    B = q.shape[0]
    dt = plan.torch_dtype
    pq = _dev(q, "q", torch.float32, qshape)
    pp = _dev(pool, "pool", dt)
    if page_table.dim() != 2 or page_table.shape[0] != B:
        raise ValueError("page_table must be [batch, max_pages]")
    pt = _dev(page_table, "page_table", torch.int32)
    psl = _dev(seq_lens, "seq_lens", torch.int32, (B,))
    prk = _dev(R_keys, "R_keys", dt)
    if R_keys.numel() != plan.key_factor_elems:
        raise ValueError(f"R_keys holds {R_keys.numel()} elements, expected {plan.key_factor_elems}")
    prv = _dev(R_value, "R_value", dt, (plan.value_rank, plan.num_kv_heads * plan.head_dim))
    if out is None:
        out = torch.empty(qshape, dtype=torch.float32, device=q.device)
    po = _dev(out, "out", torch.float32, qshape)
    need = plan.workspace_bytes(B, max_context)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    pw = _dev(workspace, "workspace", torch.uint8)
    _check(_lib.dckv_decode(plan.handle, pq, B, pp, _num_pages(plan, pool), pt, page_table.shape[1],
                            psl, int(max_context), prk, prv, po, pw, workspace.numel(),
                            _stream_handle(stream)), "decode")
    return out


def decode_noalloc(plan: Plan, q: torch.Tensor, pool: torch.Tensor, page_table: torch.Tensor,
                   seq_lens: torch.Tensor, max_context: int, R_keys: torch.Tensor,
                   R_value: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
    """decode() without a workspace: the library's fixed device scratch array
    serves instead (dckv_decode_noalloc).  `out` must be given, so that the
    call allocates nothing; calls that overlap on one GPU race."""
    Q = plan.queries_per_seq
    if q.dim() == 3 and Q == 1:
        qshape = (q.shape[0], plan.num_q_heads, plan.head_dim)
    elif q.dim() == 4:
        qshape = (q.shape[0], Q, plan.num_q_heads, plan.head_dim)
    else:
        raise ValueError("q must be [batch, Q, H_q, d_h] (or [batch, H_q, d_h] with Q = 1)")
    B = q.shape[0]
    dt = plan.torch_dtype
    pq = _dev(q, "q", torch.float32, qshape)
    pp = _dev(pool, "pool", dt)
    if page_table.dim() != 2 or page_table.shape[0] != B:
        raise ValueError("page_table must be [batch, max_pages]")
    pt = _dev(page_table, "page_table", torch.int32)
    psl = _dev(seq_lens, "seq_lens", torch.int32, (B,))
    prk = _dev(R_keys, "R_keys", dt)
    if R_keys.numel() != plan.key_factor_elems:
        raise ValueError(f"R_keys holds {R_keys.numel()} elements, expected {plan.key_factor_elems}")
    prv = _dev(R_value, "R_value", dt, (plan.value_rank, plan.num_kv_heads * plan.head_dim))
    po = _dev(out, "out", torch.float32, qshape)
    _check(_lib.dckv_decode_noalloc(plan.handle, pq, B, pp, _num_pages(plan, pool), pt,
                                    page_table.shape[1], psl, int(max_context), prk, prv, po,
                                    _stream_handle(stream)), "decode_noalloc")
    return out


def decode_rope(plan: Plan, q: torch.Tensor, pool: torch.Tensor, page_table: torch.Tensor,
                seq_lens: torch.Tensor, max_context: int, R_keys: torch.Tensor,
                R_value: torch.Tensor, rope_base: float = 10000.0,
                out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """Decode with rotary position embedding on the keys (q and the result
    [batch, H_q, d_h] fp32): key t turned by Rot(t), the query by
    Rot(seq_len - 1), planes (i, i + d_h/2) at angle pos * rope_base^(-2i/d_h)."""
    B = q.shape[0]
    qshape = (B, plan.num_q_heads, plan.head_dim)
    dt = plan.torch_dtype
    pq = _dev(q, "q", torch.float32, qshape)
    pp = _dev(pool, "pool", dt)
    if page_table.dim() != 2 or page_table.shape[0] != B:
        raise ValueError("page_table must be [batch, max_pages]")
    pt = _dev(page_table, "page_table", torch.int32)
    psl = _dev(seq_lens, "seq_lens", torch.int32, (B,))
    prk = _dev(R_keys, "R_keys", dt)
    if R_keys.numel() != plan.key_factor_elems:
        raise ValueError(f"R_keys holds {R_keys.numel()} elements, expected {plan.key_factor_elems}")
    prv = _dev(R_value, "R_value", dt, (plan.value_rank, plan.num_kv_heads * plan.head_dim))
    if out is None:
        out = torch.empty(qshape, dtype=torch.float32, device=q.device)
    po = _dev(out, "out", torch.float32, qshape)
    need = plan.rope_workspace_bytes(B, max_context)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    pw = _dev(workspace, "workspace", torch.uint8)
    _check(_lib.dckv_decode_rope(plan.handle, pq, B, pp, _num_pages(plan, pool), pt,
                                 page_table.shape[1], psl, int(max_context), prk, prv,
                                 float(rope_base), po, pw, workspace.numel(),
                                 _stream_handle(stream)), "decode_rope")
    return out


# ------------------------------------------------------ uncompressed baseline
def dense_page_elems(num_kv_heads: int, head_dim: int) -> int:
    """Elements of one page (64 tokens) of the uncompressed K/V cache."""
    n = ctypes.c_int64()
    _check(_lib.dckv_dense_page_elems(num_kv_heads, head_dim, ctypes.byref(n)), "dense_page_elems")
    return n.value


def dense_workspace_bytes(num_q_heads: int, num_kv_heads: int, head_dim: int, split_tokens: int,
                          batch: int, max_context: int) -> int:
    n = ctypes.c_size_t()
    _check(_lib.dckv_dense_workspace_bytes(num_q_heads, num_kv_heads, head_dim, split_tokens, batch,
                                           int(max_context), ctypes.byref(n)),
           "dense_workspace_bytes")
    return n.value


def dense_decode(q: torch.Tensor, kv_pool: torch.Tensor, page_table: torch.Tensor,
                 seq_lens: torch.Tensor, max_context: int, num_kv_heads: int,
                 split_tokens: int = 0, out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, events=None, stream=None) -> torch.Tensor:
    """Uncompressed decode (the baseline): q [batch, H_q, d_h] fp32 over a
    bf16 pool of pages [H_kv][64][d_h] keys then values; returns [batch, H_q,
    d_h] fp32.  `events`, a pair of torch.cuda.Event, stamp the split
    kernel's dispatch."""
    if q.dim() != 3:
        raise ValueError("q must be [batch, H_q, d_h]")
    B, Hq, d = q.shape
    pq = _dev(q, "q", torch.float32, (B, Hq, d))
    pe = dense_page_elems(num_kv_heads, d)
    pp = _dev(kv_pool, "kv_pool", torch.bfloat16)
    if kv_pool.numel() % pe:
        raise ValueError("kv_pool size is not a whole number of pages")
    if page_table.dim() != 2 or page_table.shape[0] != B:
        raise ValueError("page_table must be [batch, max_pages]")
    pt = _dev(page_table, "page_table", torch.int32)
    psl = _dev(seq_lens, "seq_lens", torch.int32, (B,))
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=q.device)
    po = _dev(out, "out", torch.float32, (B, Hq, d))
    if workspace is None:
        need = dense_workspace_bytes(Hq, num_kv_heads, d, split_tokens, B, max_context)
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    pw = _dev(workspace, "workspace", torch.uint8)
    eb = events[0].cuda_event if events else None
    ea = events[1].cuda_event if events else None
    _check(_lib.dckv_dense_decode(Hq, num_kv_heads, d, split_tokens, pq, B, pp,
                                  kv_pool.numel() // pe, pt, page_table.shape[1], psl,
                                  int(max_context), po, pw, workspace.numel(), eb, ea,
                                  _stream_handle(stream)), "dense_decode")
    return out


# ---------------------------------------------------------------- offline calls
def gram_workspace_bytes(rows: int, cols: int, center: bool = True) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.dckv_gram_workspace_bytes(int(rows), int(cols), int(bool(center)), ctypes.byref(n)),
           "gram_workspace_bytes")
    return n.value


def gram(A: torch.Tensor, center: bool = True, out: Optional[torch.Tensor] = None,
         workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """G = A~^T A~ (fp32 [cols, cols]) for samples A [rows, cols] (fp32 or
    bf16 on the GPU); A~ is A with its column means removed when `center`."""
    if A.dim() != 2:
        raise ValueError("A must be [rows, cols]")
    rows, cols = A.shape
    dt = {torch.float32: 0, torch.bfloat16: 1}.get(A.dtype)
    if dt is None:
        raise TypeError("A must be float32 or bfloat16")
    pa = _dev(A, "A", A.dtype)
    if out is None:
        out = torch.empty((cols, cols), dtype=torch.float32, device=A.device)
    po = _dev(out, "out", torch.float32, (cols, cols))
    need = gram_workspace_bytes(rows, cols, center)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=A.device)
    pw = _dev(workspace, "workspace", torch.uint8) if workspace is not None else None
    _check(_lib.dckv_gram(pa, dt, int(rows), int(cols), int(bool(center)), po, pw,
                          workspace.numel() if workspace is not None else 0, _stream_handle(stream)),
           "gram")
    return out


def head_similarity(G: torch.Tensor, num_heads: int, head_dim: int,
                    out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """S [h, h] fp32 from a centred Gram G [h*d_h, h*d_h] of per-head activations."""
    n = num_heads * head_dim
    pg = _dev(G, "G", torch.float32, (n, n))
    if out is None:
        out = torch.empty((num_heads, num_heads), dtype=torch.float32, device=G.device)
    ps = _dev(out, "out", torch.float32, (num_heads, num_heads))
    _check(_lib.dckv_head_similarity(pg, int(num_heads), int(head_dim), ps, _stream_handle(stream)),
           "head_similarity")
    return out


def cluster_heads(S, K: int):
    """Group id of every head (host call): average-linkage clustering of 1 - S."""
    import numpy as np
    Sd = np.ascontiguousarray(np.asarray(S, dtype=np.float64))
    h = Sd.shape[0]
    if Sd.shape != (h, h):
        raise ValueError("S must be square")
    out = (ctypes.c_int32 * h)()
    _check(_lib.dckv_cluster_heads(Sd.ctypes.data_as(ctypes.c_void_p), h, int(K), out), "cluster_heads")
    return list(out)


def cluster_merges(S):
    """The clustering's whole merge sequence (host call): a list of
    (a, b, height) -- clusters named by their smallest head, a < b, merged at
    average-linkage distance `height` -- h - 1 entries in merge order."""
    import numpy as np
    Sd = np.ascontiguousarray(np.asarray(S, dtype=np.float64))
    h = Sd.shape[0]
    if Sd.shape != (h, h):
        raise ValueError("S must be square")
    n = max(h - 1, 1)
    ma, mb = (ctypes.c_int32 * n)(), (ctypes.c_int32 * n)()
    ht = (ctypes.c_double * n)()
    _check(_lib.dckv_cluster_merges(Sd.ctypes.data_as(ctypes.c_void_p), h, ma, mb,
                                    ctypes.cast(ht, ctypes.c_void_p)), "cluster_merges")
    return [(ma[i], mb[i], ht[i]) for i in range(h - 1)]


def allocate_ranks(heads: Sequence[int], energy: Sequence[float], energy_total: float,
                   sigmas: Sequence, rank_cap: Sequence[int], r: int):
    """(init_ranks, ranks) of the energy rule and the greedy budget step (host call)."""
    import numpy as np
    K = len(heads)
    stride = max(len(s) for s in sigmas)
    sig = np.zeros((K, stride))
    for i, s in enumerate(sigmas):
        sig[i, :len(s)] = np.asarray(s, dtype=np.float64)
    en = np.ascontiguousarray(np.asarray(energy, dtype=np.float64))
    init = (ctypes.c_int32 * K)()
    ranks = (ctypes.c_int32 * K)()
    _check(_lib.dckv_allocate_ranks(K, _i32_array(heads), en.ctypes.data_as(ctypes.c_void_p),
                                    float(energy_total), sig.ctypes.data_as(ctypes.c_void_p), stride,
                                    _i32_array(rank_cap), int(r), init, ranks), "allocate_ranks")
    return list(init), list(ranks)
