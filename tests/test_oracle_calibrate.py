"""Pins of the value-calibration oracle (Sec. III-D): each closed-form update
against a library least-squares solve, zero gradients, the error ordering the
paper states, and the isotropic and full-rank special cases."""

import numpy as np
import pytest

from oracle import calibrate as ocal


def _problem(seed, m=24, n=20, N=200, aniso=True):
    g = np.random.default_rng(seed)
    W = g.standard_normal((m, n))
    X = g.standard_normal((N, m))
    if aniso:
        X = X * np.logspace(0, 1.5, m)[None, :]     # calibration inputs with uneven scales
    return X, W


def test_right_update_is_the_least_squares_solution():
    X, W = _problem(1)
    L, _ = ocal.svd_factors(W, 6)
    R = ocal.update_right(ocal.gram(X), W, L)
    R_ls = np.linalg.lstsq(X @ L, X @ W, rcond=None)[0]       # min ||(X L) R - X W||
    assert np.allclose(R, R_ls, rtol=1e-8, atol=1e-10)
    # gradient of eps with respect to R vanishes: L^T X^T (X L R - X W) = 0
    grad = L.T @ X.T @ (X @ L @ R - X @ W)
    assert np.max(np.abs(grad)) <= 1e-8 * np.max(np.abs(L.T @ X.T @ X @ W))


def test_left_update_is_the_least_squares_solution():
    X, W = _problem(2)
    _, R = ocal.svd_factors(W, 5)
    L = ocal.update_left(W, R)
    Lt_ls = np.linalg.lstsq(R.T, W.T, rcond=None)[0]           # min ||L R - W||
    assert np.allclose(L, Lt_ls.T, rtol=1e-8, atol=1e-10)
    # with X of full column rank this also zeroes d eps / d L = X^T (X L R - X W) R^T
    grad = X.T @ (X @ L @ R - X @ W) @ R.T
    assert np.max(np.abs(grad)) <= 1e-8 * np.max(np.abs(X.T @ X @ W @ R.T))


def test_refinement_never_increases_the_calibration_error():
    for seed in range(5):
        X, W = _problem(10 + seed)
        for r in (2, 7, 15):
            out = ocal.refine(X, W, r)
            assert out["eps_mid"] <= out["eps_svd"] * (1 + 1e-12)
            assert out["eps"] <= out["eps_mid"] * (1 + 1e-12)
    # uneven calibration scales: a strict gain over plain SVD
    X, W = _problem(3)
    out = ocal.refine(X, W, 6)
    assert out["eps"] < 0.9 * out["eps_svd"]


def test_isotropic_calibration_keeps_the_svd_factors():
    # G = c^2 I: the SVD factors already minimise eps, and the R update returns them
    g = np.random.default_rng(4)
    m, n, r = 16, 12, 5
    W = g.standard_normal((m, n))
    Q, _ = np.linalg.qr(g.standard_normal((m, m)))
    X = 2.5 * Q                                                  # X^T X = 6.25 I
    out = ocal.refine(X, W, r)
    assert np.allclose(out["R_mid"], out["R_svd"], atol=1e-10)
    assert out["eps"] == pytest.approx(out["eps_svd"], rel=1e-10)


def test_full_rank_has_zero_error():
    X, W = _problem(5, m=10, n=8)
    out = ocal.refine(X, W, 8)
    assert out["eps"] <= 1e-18 * np.sum((X @ W) ** 2)


def test_calibration_error_definition():
    # eps on a hand-sized case: X = I reduces eps to ||L R - W||_F^2
    W = np.array([[3.0, 0.0], [0.0, 1.0]])
    L, R = ocal.svd_factors(W, 1)
    assert ocal.calib_error(np.eye(2), W, L, R) == pytest.approx(1.0, abs=1e-12)
