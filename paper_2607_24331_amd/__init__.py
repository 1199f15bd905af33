"""DynaCalKV compressed-KV decode attention on MI355X (gfx950).

The hot path -- latent append and decode -- runs in hand-written HIP kernels
behind the C ABI of include/dckv.h (libdckv.so).  Importing this package
loads that library and fails if it has not been built.
"""

from .dckv import (DckvError, Plan, allocate_ranks, cluster_heads, cluster_merges, decode,  # noqa: F401
                   decode_noalloc, decode_rope, dense_decode, dense_page_elems, dense_workspace_bytes, gram,
                   gram_workspace_bytes, head_similarity, latent_append)
from . import capi  # noqa: F401

__all__ = ["Plan", "latent_append", "decode", "decode_noalloc", "decode_rope", "dense_decode", "dense_page_elems", "DckvError", "capi",
           "gram", "gram_workspace_bytes", "head_similarity", "cluster_heads", "cluster_merges", "allocate_ranks"]
