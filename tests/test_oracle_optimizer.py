"""Pins of the M-FAC optimizer oracle (Section 4.2, Application 2)."""

import numpy as np

from oracle.optimizer import MFACOracle


def test_window_of_one_is_sherman_morrison():
    """m = 1: F = lam I + v v^T, so F^-1 v = v / (lam + |v|^2) (closed form)."""
    rng = np.random.default_rng(0)
    d, lam, lr = 50, 0.3, 0.7
    w = rng.standard_normal(d)
    opt = MFACOracle(d, 1, lam)
    for _ in range(3):
        g = rng.standard_normal(d)
        v = g.astype(np.float32).astype(np.float64)
        w_next, y = opt.step(w, g, lr)
        np.testing.assert_allclose(y, v / (lam + v @ v), rtol=1e-12)
        np.testing.assert_allclose(w_next, w - lr * v / (lam + v @ v), rtol=1e-12)
        w = w_next


def test_trajectory_matches_dense_solve_over_explicit_window():
    """F_t built densely from a list of the last m inserted vectors (zero rows
    before the window is full), weight decay and per-coordinate lr."""
    rng = np.random.default_rng(1)
    d, m, lam, steps = 30, 4, 0.2, 9
    lr = np.where(np.arange(d) < 20, 0.1, 0.05)
    wd = np.where(np.arange(d) < 20, 0.01, 0.0)
    w_o = rng.standard_normal(d)
    w_d = w_o.copy()
    opt = MFACOracle(d, m, lam)
    recent = []
    for _ in range(steps):
        g = rng.standard_normal(d)
        w_o, _ = opt.step(w_o, g, lr, wd)
        v = (g + wd * w_d).astype(np.float32).astype(np.float64)
        recent = (recent + [v])[-m:]
        F = lam * np.eye(d) + sum(np.outer(r, r) for r in recent) / m
        w_d = w_d - lr * np.linalg.solve(F, v)
        np.testing.assert_allclose(w_o, w_d, rtol=1e-10, atol=1e-12)


def test_weight_decay_enters_the_window():
    rng = np.random.default_rng(2)
    d, wd = 12, 0.5
    w = rng.standard_normal(d)
    g = rng.standard_normal(d)
    opt = MFACOracle(d, 3, 1.0)
    opt.step(w, g, 0.1, wd)
    np.testing.assert_array_equal(opt.window.G[0], (g + wd * w).astype(np.float32))
    assert np.all(opt.window.G[1:] == 0)
