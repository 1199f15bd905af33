"""Parameter counts of the compressed key projection (Sec. III-C).

All counts are exact integers or Fractions.

  group_factor_params   sum over groups of m r_i + r_i h_i d_h
                        (left side of the per-layer count equations)
  identity_rhs          m r + n * sum(r_i alpha_i), valid when sum r_i = r
  final_params          m * sum(r_i) + n * sum(r_i alpha_i), the count after
                        the greedy rank adjustment (sum r_i may fall below r)
  fixed_group_params    m r + r n 4 / h: fixed groups of four heads with the
                        uniform rank r / K, K = h / 4 (the ReCalKV baseline)
  budget_holds          sum(r_i alpha_i) <= 4 r / h, the budget inequality
"""

from __future__ import annotations

from fractions import Fraction
from typing import Sequence


def group_factor_params(m: int, ranks: Sequence[int], heads: Sequence[int], head_dim: int) -> int:
    return sum(m * r + r * h * head_dim for r, h in zip(ranks, heads))


def weighted_rank(ranks: Sequence[int], heads: Sequence[int]) -> Fraction:
    """sum_i r_i alpha_i with alpha_i = h_i / h."""
    h = sum(heads)
    return sum((Fraction(r * hi, h) for r, hi in zip(ranks, heads)), Fraction(0))


def identity_rhs(m: int, r: int, n: int, ranks: Sequence[int], heads: Sequence[int]) -> Fraction:
    return m * r + n * weighted_rank(ranks, heads)


def final_params(m: int, n: int, ranks: Sequence[int], heads: Sequence[int]) -> Fraction:
    return m * sum(ranks) + n * weighted_rank(ranks, heads)


def fixed_group_params(m: int, r, n: int, h: int) -> Fraction:
    return m * Fraction(r) + Fraction(r) * n * Fraction(4, h)


def budget_holds(ranks: Sequence[int], heads: Sequence[int], r: int) -> bool:
    h = sum(heads)
    return weighted_rank(ranks, heads) <= Fraction(4 * r, h)


def fixed_group_baseline_ranks(r: int, h: int):
    """Uniform ranks of the fixed four-head grouping: K = h/4 groups of r/K.

    When r/K is not an integer the ranks differ by at most one, the larger
    ones first (a stated reading; the paper only states r_i = r/K)."""
    K = h // 4
    base, extra = divmod(r, K)
    return [base + (1 if i < extra else 0) for i in range(K)], [4] * K
