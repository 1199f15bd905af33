"""Pins of the oracle's fp64 -> bf16 round-to-nearest-even."""

import numpy as np
import pytest
import torch

from oracle.bf16 import round_to_bf16, ulp_bf16


def _bits(v: float) -> int:
    """Bit pattern of a value that is exactly a bf16 value."""
    u = np.array([v], dtype=np.float32).view(np.uint32)[0]
    assert u & 0xFFFF == 0
    return int(u >> 16)


@pytest.mark.parametrize("v, expect_bits", [
    (1.0, 0x3F80),
    (-2.0, 0xC000),
    (np.pi, 0x4049),                    # 3.140625
    (0.1, 0x3DCD),                      # 0.10009765625
    (65504.0, 0x4780),                  # 65536 after rounding: 65504 = 1.999 * 2^15
    (1.0 + 2.0 ** -8, 0x3F80),          # tie between 1 and 1+2^-7: even is 1
    (1.0 + 3 * 2.0 ** -8, 0x3F82),      # tie between 1+2^-7 and 1+2^-6: even is 1+2^-6
    (1.0 + 2.0 ** -8 + 2.0 ** -40, 0x3F81),  # just above the tie
    (-(1.0 + 2.0 ** -8), 0xBF80),
])
def test_hand_picked_patterns(v, expect_bits):
    r = float(round_to_bf16(np.array([v]))[0])
    assert _bits(r) == expect_bits


def test_rounds_once_from_fp64():
    # 1 + 2^-8 + 2^-30 lies above the tie, so the nearest bf16 is 1 + 2^-7.
    # Going through fp32 first would drop 2^-30, land on the tie and give 1.
    v = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert float(round_to_bf16(np.array([v]))[0]) == 1.0 + 2.0 ** -7
    via_f32 = torch.tensor([v], dtype=torch.float32).to(torch.bfloat16).item()
    assert via_f32 == 1.0


def test_range_ends():
    max_finite = (2.0 - 2.0 ** -7) * 2.0 ** 127
    r = round_to_bf16(np.array([max_finite, (2.0 - 2.0 ** -8) * 2.0 ** 127, -1e39,
                                2.0 ** -133, 2.0 ** -134, 1.5 * 2.0 ** -134, 2.0 ** -126 * 1.00390625]))
    assert r[0] == max_finite
    assert np.isinf(r[1]) and r[1] > 0          # tie at the top rounds to even = overflow
    assert np.isinf(r[2]) and r[2] < 0
    assert r[3] == 2.0 ** -133                  # smallest subnormal is exact
    assert r[4] == 0.0                          # tie between 0 and 2^-133: even is 0
    assert r[5] == 2.0 ** -133
    assert r[6] == 2.0 ** -126                  # normal range near the bottom


def test_special_values_pass_through():
    r = round_to_bf16(np.array([0.0, -0.0, np.inf, -np.inf, np.nan]))
    assert r[0] == 0.0 and r[1] == 0.0 and np.signbit(r[1])
    assert np.isposinf(r[2]) and np.isneginf(r[3]) and np.isnan(r[4])


def test_matches_library_on_fp32_inputs():
    # For inputs that are fp32 values, one rounding from fp64 equals the
    # library's fp32 -> bf16 round-to-nearest-even conversion.
    g = np.random.default_rng(7)
    mant = g.standard_normal(200_000).astype(np.float32)
    scale = np.exp2(g.integers(-140, 127, size=mant.size)).astype(np.float32)
    with np.errstate(over="ignore"):
        v = (mant * scale).astype(np.float32)
    v = v[np.isfinite(v)]
    ours = round_to_bf16(v.astype(np.float64))
    lib = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    same = (ours == lib) | (np.isnan(ours) & np.isnan(lib))
    assert same.all(), v[~same][:10]


def test_error_within_half_ulp():
    g = np.random.default_rng(3)
    v = g.standard_normal(100_000) * np.exp2(g.integers(-30, 30, 100_000))
    r = round_to_bf16(v)
    assert np.all(np.abs(r - v) <= 0.5 * ulp_bf16(r) * (1 + 1e-12))
