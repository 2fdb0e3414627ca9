"""Explicit d x d damped empirical Fisher, for tiny d (test infrastructure only).

F = lambda * I_d + (1/m) * sum_i g_i g_i^T  (Theorem 1, with the sum over the
whole window; Section 2 eq. 1 gives the undamped empirical Fisher).
The inverse-vector product and the inverse diagonal are taken with dense LAPACK
solves on the formed matrix, which is what "the direct computation" means.
"""

import numpy as np


def fisher(G, lam, m=None):
    """Dense F for the rows of G (m x d). ``m`` is the 1/m scale (capacity)."""
    G = np.asarray(G, dtype=np.float64)
    mm = G.shape[0] if m is None else m
    d = G.shape[1]
    return lam * np.eye(d) + (G.T @ G) / mm


def ihvp(G, lam, X, m=None):
    """F^-1 X by a dense solve; X is (d,) or (n, d)."""
    F = fisher(G, lam, m)
    X = np.asarray(X, dtype=np.float64)
    return np.linalg.solve(F, X.T).T


def inv_diag(G, lam, m=None):
    F = fisher(G, lam, m)
    return np.diag(np.linalg.inv(F)).copy()


def woodbury_recursive_inverse(G, lam, m=None):
    """F^-1 by the rank-one Sherman-Morrison recursion of Section 2 eq. 2.

    Starts from lambda^-1 I and folds the rows in one at a time; with the 1/m
    scale of Theorem 1 the denominator is m + g^T F_{i-1}^-1 g.
    """
    G = np.asarray(G, dtype=np.float64)
    mm = G.shape[0] if m is None else m
    d = G.shape[1]
    Finv = np.eye(d) / lam
    for g in G:
        v = Finv @ g
        Finv = Finv - np.outer(v, v) / (mm + g @ v)
    return Finv
