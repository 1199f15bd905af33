"""Pins of the oracle's latent write z = x L (Sec. III-A), rounded once."""

import numpy as np

from oracle import append, bf16, layout


def test_one_hot_rows_select_factor_rows():
    g = np.random.default_rng(0)
    m, RK, rv = 12, 5, 3
    Lk = g.standard_normal((m, RK))
    Lv = g.standard_normal((m, rv))
    x = np.zeros((m, m))
    x[np.arange(m), (np.arange(m) * 5) % m] = 1.0
    Zk, Zv = append.latents(x, Lk, Lv, "bf16")
    np.testing.assert_array_equal(Zk, bf16.round_to_bf16(Lk[(np.arange(m) * 5) % m]))
    np.testing.assert_array_equal(Zv, bf16.round_to_bf16(Lv[(np.arange(m) * 5) % m]))


def test_small_integers_are_exact():
    g = np.random.default_rng(1)
    x = g.integers(-3, 4, size=(20, 16)).astype(np.float64)
    L = g.integers(-3, 4, size=(16, 9)).astype(np.float64)
    Zk, _ = append.latents(x, L, L[:, :2], "bf16")
    ref = np.zeros((20, 9))
    for i in range(20):
        for j in range(9):
            ref[i, j] = sum(x[i, k] * L[k, j] for k in range(16))   # |.| <= 144: exact in bf16
    np.testing.assert_array_equal(Zk, ref)


def test_rounding_is_nearest_and_single():
    g = np.random.default_rng(2)
    x = g.standard_normal((50, 64))
    L = g.standard_normal((64, 7)) / 8
    Zk, _ = append.latents(x, L, L, "bf16")
    exact = x @ L
    assert np.all(np.abs(Zk - exact) <= 0.5 * bf16.ulp_bf16(Zk) * (1 + 1e-12))
    Z32, _ = append.latents(x, L, L, "f32")
    np.testing.assert_array_equal(Z32, exact.astype(np.float32).astype(np.float64))


def test_append_places_tokens_after_existing_ones():
    g = np.random.default_rng(3)
    m, RK, rv = 8, 6, 4
    Lk, Lv = g.standard_normal((m, RK)), g.standard_normal((m, rv))
    table = np.array([[2, 0, 1]], dtype=np.int32)
    pool = layout.new_pool(3, RK, rv)
    x1, x2 = g.standard_normal((70, m)), g.standard_normal((60, m))
    append.append(pool, table, 0, 0, x1, Lk, Lv, "bf16")
    append.append(pool, table, 0, 70, x2, Lk, Lv, "bf16")
    Zk, Zv = layout.unpack(pool, table, 0, 130, RK, rv)
    Zk_ref, Zv_ref = append.latents(np.vstack([x1, x2]), Lk, Lv, "bf16")
    np.testing.assert_array_equal(Zk, Zk_ref)
    np.testing.assert_array_equal(Zv, Zv_ref)
