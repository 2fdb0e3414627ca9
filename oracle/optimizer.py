"""M-FAC preconditioned SGD on a flat weight vector, float64 (test infrastructure only).

Definition followed (Section 4.2, Application 2: matrix-free preconditioned
SGD; no momentum, as in the paper's optimizer runs):
    v_t     = g_t + wd * w_t                       (coupled weight decay, 0 by default)
    F_t     = lambda * I + (1/m) * sum of v v^T over the last m vectors v
              (the oldest is dropped; before m steps the missing ones are zero rows)
    w_{t+1} = w_t - lr * F_t^-1 v_t
lr and wd may be scalars or per-coordinate arrays (parameter groups). The
vector entering the window is stored in fp32, as the window holds fp32
gradients; F_t^-1 v_t is evaluated in float64 by the window oracle.
Pinned in tests/test_oracle_optimizer.py: the m = 1 Sherman-Morrison closed
form, a dense d x d solve over an explicit list of the last m vectors, and
the weight-decay term entering the window.
"""

import numpy as np

from .dynamic import WindowOracle


class MFACOracle:
    def __init__(self, d, m, lam):
        self.window = WindowOracle(d, m, lam)

    def step(self, w, g, lr, wd=0.0):
        """One step from weights w with loss gradient g; returns (w_next, F^-1 v)."""
        w = np.asarray(w, np.float64)
        v = np.asarray(g, np.float64) + np.asarray(wd, np.float64) * w
        y = self.window.slide(v.astype(np.float32))
        return w - np.asarray(lr, np.float64) * y, y
