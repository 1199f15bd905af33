"""The seeded workloads have the stated shapes and are reproducible."""

import numpy as np
import pytest

from workloads import WORKLOAD_NAMES, make_workload
from workloads.inputs import make_inputs, make_page_table


@pytest.mark.parametrize("name", WORKLOAD_NAMES)
def test_stated_shapes(name):
    wl = make_workload(name)
    assert sum(wl.group_sizes) == wl.num_kv_heads
    assert len(wl.group_of_kv) == wl.num_kv_heads
    assert all(1 <= r <= s * wl.head_dim for r, s in zip(wl.group_rank, wl.group_sizes))
    assert wl.num_q_heads % wl.num_kv_heads == 0
    assert len(wl.seq_lens) == wl.batch
    assert wl.prefill_lens[0] + wl.append_tokens == wl.seq_lens[0]
    expect = {
        "tiny_mha_f32": (2, 128, 128, (4, 4)),
        "mha7b_b8_t4k": (8, 2048, 2048, (2, 3, 4, 4, 5, 6, 4, 4)),
        "gqa8b_b4_t32k": (3, 768, 768, (2, 3, 3)),
        "mha_long_t128k": (6, 1536, 2048, (8, 6, 6, 5, 4, 3)),
        "mha_ragged_b64": (10, 1228, 1536, None),
    }[name]
    assert wl.num_groups == expect[0]
    assert wl.key_rank_total == expect[1]
    assert wl.value_rank == expect[2]
    if expect[3] is not None:
        assert wl.group_sizes == expect[3]


def test_ragged_lengths_and_pages():
    wl = make_workload("mha_ragged_b64")
    assert all(1024 <= t <= 8192 for t in wl.seq_lens)
    table = make_page_table(wl)
    used = np.concatenate([table[b, :n] for b, n in enumerate(wl.pages_per_seq)])
    assert np.array_equal(np.sort(used), np.arange(wl.total_pages))
    assert not np.array_equal(used, np.arange(wl.total_pages))   # physically shuffled


def test_reproducible_small():
    wl = make_workload("tiny_mha_f32")
    a, b = make_inputs(wl), make_inputs(wl)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.R_value, b.R_value)
    assert a.x.shape == (256, 512) and a.q.shape == (1, 8, 64)
    assert [blk.shape for blk in a.R_blocks] == [(48, 256), (80, 256)]


def test_orthonormal_rows_before_rounding():
    from workloads.inputs import _orthonormal_rows
    g = np.random.default_rng(0)
    R = _orthonormal_rows(g, 40, 128)
    np.testing.assert_allclose(R @ R.T, np.eye(40), atol=1e-12)
