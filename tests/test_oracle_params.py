"""Pins of the key-factor parameter counts (Sec. III-C) and the budget
reading used by the workloads."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import params

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_k_params.json")


def test_tiny_layer_counts_equal_fixed_grouping():
    # 8 heads x 64, m = 512, groups of four heads with ranks 48 and 80 (sum 128):
    # both the group count and the fixed four-head baseline give 98,304, and the
    # budget inequality holds with equality (sum r_i alpha_i = 64 = 4 r / h).
    m, d, h, ranks, heads = 512, 64, 8, [48, 80], [4, 4]
    n = h * d
    assert params.group_factor_params(m, ranks, heads, d) == 98304
    assert params.fixed_group_params(m, 128, n, h) == 98304
    assert params.weighted_rank(ranks, heads) == 64
    assert params.budget_holds(ranks, heads, 128)


def test_identity_holds_exactly_for_random_partitions():
    # sum_i [m r_i + r_i h_i d_h] = m r + n sum_i r_i alpha_i whenever sum r_i = r.
    g = np.random.default_rng(11)
    for _ in range(500):
        h = int(g.integers(1, 40))
        d = int(g.choice([16, 64, 128]))
        m = int(g.integers(1, 5000))
        K = int(g.integers(1, h + 1))
        cuts = np.sort(g.choice(np.arange(1, h), size=K - 1, replace=False)) if K > 1 else []
        heads = np.diff(np.concatenate([[0], cuts, [h]])).astype(int).tolist()
        ranks = [int(g.integers(1, hi * d + 1)) for hi in heads]
        r = sum(ranks)
        lhs = params.group_factor_params(m, ranks, heads, d)
        assert Fraction(lhs) == params.identity_rhs(m, r, h * d, ranks, heads)
        assert Fraction(lhs) == params.final_params(m, h * d, ranks, heads)


def test_uniform_four_head_grouping_is_the_baseline():
    # With groups of four heads and equal ranks r/K the group count reduces to
    # m r + r n 4 / h.
    for h, d, m, per in [(8, 64, 2048, 12), (16, 128, 2048, 30), (32, 64, 2048, 7)]:
        K = h // 4
        ranks, heads = [per] * K, [4] * K
        assert params.group_factor_params(m, ranks, heads, d) == params.fixed_group_params(m, per * K, h * d, h)


def test_table1_differences_reproduce():
    with open(GOLDEN) as f:
        rows = json.load(f)["models"]
    for row in rows:
        diff = row["fixed_group"] - row["dynamic"]
        assert diff == row["difference"]
        pct = Fraction(diff * 100, row["fixed_group"])
        assert f"{float(pct):.2f}" == row["percent"]


def test_table1_fixed_group_totals_fit_baseline_formula():
    # Summed over layers, the baseline count is (m + 4 n / h) * sum_l r_l.  With
    # the inferred hidden size m = 2048 every printed total is an integer
    # multiple of m + 4 n / h; a wrong factor (4 h / n, n / 4 h, a dropped m)
    # breaks this for at least one model.
    with open(GOLDEN) as f:
        rows = json.load(f)["models"]
    m = 2048
    expect_rank_sums = {"Llama-3.2-1B-Instruct": 1568, "Qwen1.5-1.8B-Chat": 11712,
                        "SmolLM2-1.7B-Instruct": 14752}
    for row in rows:
        unit = params.fixed_group_params(m, 1, row["kv_dim"], row["heads"])
        total = Fraction(row["fixed_group"])
        q = total / unit
        assert q.denominator == 1
        assert q == expect_rank_sums[row["model"]]
        assert params.fixed_group_params(m, int(q), row["kv_dim"], row["heads"]) == total


def test_budget_reading_for_workloads():
    # The GQA workload's ranks {192,256,320} on groups {2,3,3} of 8 heads stay
    # within the budget (sum r alpha = 264 <= 4 * 768 / 8 = 384).
    assert params.weighted_rank([192, 256, 320], [2, 3, 3]) == 264
    assert params.budget_holds([192, 256, 320], [2, 3, 3], 768)
    # Size-proportional ranks on unequal groups exceed it (Cauchy-Schwarz):
    # nominal 48 h_g on {8,6,6,5,4,3} gives 279 > 192.
    heads = [8, 6, 6, 5, 4, 3]
    assert params.weighted_rank([48 * x for x in heads], heads) == Fraction(279)
    assert not params.budget_holds([48 * x for x in heads], heads, 1536)


def test_baseline_ranks_split_nonintegral_budget():
    ranks, heads = params.fixed_group_baseline_ranks(1228, 32)
    assert sum(ranks) == 1228 and heads == [4] * 8
    assert sorted(set(ranks)) == [153, 154]
