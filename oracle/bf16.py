"""Rounding of fp64 values to bfloat16, round-to-nearest, ties to even.

bfloat16 keeps 8 significant bits (7 stored) and the fp32 exponent range:
largest finite value (2 - 2^-7) * 2^127, smallest normal 2^-126, smallest
subnormal 2^-133.  The rounding is done from fp64 in one step (never through
fp32, which would round twice).  The paper fixes no storage precision; bf16
latents with round-to-nearest-even are a stated reading.
"""

from __future__ import annotations

import numpy as np

_MIN_EXP_QUANTUM = -133          # exponent of the smallest subnormal
_MAX_FINITE = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_to_bf16(v) -> np.ndarray:
    """Nearest bf16 value of each fp64 input (ties to even), as fp64."""
    v = np.asarray(v, dtype=np.float64)
    out = np.array(v, copy=True)
    finite = np.isfinite(v) & (v != 0.0)
    x = v[finite]
    # x = f * 2^e with 0.5 <= |f| < 1; bf16 spacing in [2^(e-1), 2^e) is 2^(e-8)
    _, e = np.frexp(x)
    qexp = np.maximum(e - 8, _MIN_EXP_QUANTUM)
    scaled = np.ldexp(x, -qexp)               # exact: only the exponent changes
    r = np.ldexp(np.rint(scaled), qexp)       # np.rint rounds half to even
    r = np.where(np.abs(r) > _MAX_FINITE, np.copysign(np.inf, x), r)
    out[finite] = r
    return out


def round_to_f32(v) -> np.ndarray:
    """Nearest fp32 value (ties to even) of each fp64 input, as fp64."""
    return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_storage(v, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(v)
    if dtype == "f32":
        return round_to_f32(v)
    raise ValueError(dtype)


def ulp_bf16(v) -> np.ndarray:
    """Spacing of bf16 values at |v| (the gap above the bf16 value nearest v)."""
    v = np.abs(np.asarray(v, dtype=np.float64))
    _, e = np.frexp(np.where(v == 0, 2.0 ** -126, v))
    return np.ldexp(1.0, np.maximum(e - 8, _MIN_EXP_QUANTUM))
