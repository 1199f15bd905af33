"""DynaCalKV compressed-KV decode attention on MI355X (gfx950).

The hot path -- latent append and decode -- runs in hand-written HIP kernels
behind the C ABI of include/dckv.h (libdckv.so).  Importing this package
loads that library and fails if it has not been built.
"""

from .dckv import (DckvError, Plan, decode, dense_decode, dense_page_elems,  # noqa: F401
                   dense_workspace_bytes, latent_append)
from . import capi  # noqa: F401

__all__ = ["Plan", "latent_append", "decode", "dense_decode", "dense_page_elems", "DckvError", "capi"]
