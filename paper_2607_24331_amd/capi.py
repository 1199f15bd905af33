"""ctypes declarations of the C ABI in include/dckv.h (libdckv.so).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any entry point.
"""

from __future__ import annotations

import ctypes
import os
import re

# DCKV_LIBRARY selects another build of the same library (the sanitized one)
LIB_PATH = os.environ.get("DCKV_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                          "libdckv.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "include", "dckv.h")

DCKV_OK = 0
DCKV_EINVAL = -1
DCKV_EDTYPE = -2
DCKV_EALIGN = -3
DCKV_EWORKSPACE = -4
DCKV_EHIP = -5
DCKV_ENOMEM = -6
DCKV_F32 = 0
DCKV_BF16 = 1
PAGE_TOKENS = 64
NOALLOC_SCRATCH_BYTES = 64 << 20

STATUS_NAMES = {0: "DCKV_OK", -1: "DCKV_EINVAL", -2: "DCKV_EDTYPE", -3: "DCKV_EALIGN",
                -4: "DCKV_EWORKSPACE", -5: "DCKV_EHIP", -6: "DCKV_ENOMEM"}


class LayerDesc(ctypes.Structure):
    _fields_ = [
        ("hidden", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("num_groups", ctypes.c_int32),
        ("group_of_kv_head", ctypes.POINTER(ctypes.c_int32)),
        ("group_rank", ctypes.POINTER(ctypes.c_int32)),
        ("value_rank", ctypes.c_int32),
        ("latent_dtype", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("head_slices", ctypes.c_int32),
        ("queries_per_seq", ctypes.c_int32),
        ("decode_waves", ctypes.c_int32),
        ("decode_passes", ctypes.c_int32),
    ]


class PlanGeometry(ctypes.Structure):
    _fields_ = [
        ("key_rank_total", ctypes.c_int32),
        ("key_width_padded", ctypes.c_int32),
        ("value_width_padded", ctypes.c_int32),
        ("value_rank", ctypes.c_int32),
        ("q_per_kv", ctypes.c_int32),
        ("folded_query_len", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("mfma_path", ctypes.c_int32),
        ("head_slices", ctypes.c_int32),
        ("queries_per_seq", ctypes.c_int32),
        ("decode_waves", ctypes.c_int32),
        ("decode_ring", ctypes.c_int32),
        ("value_tiles_per_wave", ctypes.c_int32),
        ("key_chunk_loads", ctypes.c_int32),
        ("two_pass", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("page_elems", ctypes.c_int64),
        ("value_base", ctypes.c_int64),
        ("key_factor_elems", ctypes.c_int64),
    ]


class LaunchInfo(ctypes.Structure):
    _fields_ = [
        ("kernels", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("n_split", ctypes.c_int32),
        ("head_slices", ctypes.c_int32),
        ("value_tiles", ctypes.c_int32),
    ]


_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pi64 = ctypes.POINTER(ctypes.c_int64)

SIGNATURES = {
    "dckv_plan_create": (ctypes.c_int, [ctypes.POINTER(LayerDesc), ctypes.POINTER(_vp)]),
    "dckv_plan_destroy": (None, [_vp]),
    "dckv_plan_info": (ctypes.c_int, [_vp, ctypes.POINTER(PlanGeometry), _pi32, _pi32, _pi32, _pi64]),
    "dckv_decode_workspace_bytes": (ctypes.c_int, [_vp, _i32, _i32, ctypes.POINTER(ctypes.c_size_t)]),
    "dckv_decode_launch_info": (ctypes.c_int, [_vp, _i32, _i32, ctypes.POINTER(LaunchInfo)]),
    "dckv_latent_append": (ctypes.c_int, [_vp, _vp, _i32, _vp, _vp, _vp, _vp, _i64, _vp]),
    "dckv_decode": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i64, _vp, _i32, _vp, _i32, _vp, _vp, _vp,
                                   _vp, ctypes.c_size_t, _vp]),
    "dckv_decode_noalloc": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i64, _vp, _i32, _vp, _i32, _vp,
                                           _vp, _vp, _vp]),
    "dckv_plan_set_profile_events": (ctypes.c_int, [_vp, _vp, _vp]),
    "dckv_rope_workspace_bytes": (ctypes.c_int, [_vp, _i32, _i32, ctypes.POINTER(ctypes.c_size_t)]),
    "dckv_decode_rope": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i64, _vp, _i32, _vp, _i32, _vp, _vp,
                                        ctypes.c_double, _vp, _vp, ctypes.c_size_t, _vp]),
    "dckv_dense_page_elems": (ctypes.c_int, [_i32, _i32, ctypes.POINTER(ctypes.c_int64)]),
    "dckv_dense_workspace_bytes": (ctypes.c_int, [_i32, _i32, _i32, _i32, _i32, _i32,
                                                  ctypes.POINTER(ctypes.c_size_t)]),
    "dckv_dense_decode": (ctypes.c_int, [_i32, _i32, _i32, _i32, _vp, _i32, _vp, _i64, _vp, _i32,
                                         _vp, _i32, _vp, _vp, ctypes.c_size_t, _vp, _vp, _vp]),
    "dckv_gram_workspace_bytes": (ctypes.c_int, [_i64, _i32, _i32, ctypes.POINTER(ctypes.c_size_t)]),
    "dckv_gram": (ctypes.c_int, [_vp, _i32, _i64, _i32, _i32, _vp, _vp, ctypes.c_size_t, _vp]),
    "dckv_head_similarity": (ctypes.c_int, [_vp, _i32, _i32, _vp, _vp]),
    "dckv_cluster_merges": (ctypes.c_int, [_vp, _i32, _pi32, _pi32, _vp]),
    "dckv_cluster_heads": (ctypes.c_int, [_vp, _i32, _i32, _pi32]),
    "dckv_allocate_ranks": (ctypes.c_int, [_i32, _pi32, _vp, ctypes.c_double, _vp, _i32, _pi32, _i32,
                                           _pi32, _pi32]),
    "dckv_last_error": (ctypes.c_char_p, []),
}


def header_functions(path: str = HEADER_PATH):
    """Names of the functions include/dckv.h declares."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dckv_[a-z_]+)\s*\(", text)))


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build it with `python paper_2607_24331_amd/build.py` "
            "(the decode and append paths have no fallback)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib
