"""The paper's own recursions, in float64 (test infrastructure only).

These follow the algorithms' steps in the paper's order and notation, written
from the equations (0-based indices here, 1-based in the paper). They are the
cross-check O1'/O2' of the plain-definition oracles in dynamic.py/static.py.

Readings taken where the printed text is garbled or silent:
  * Algorithm 1 (Appendix B): iteration i subtracts the outer product of the
    single row D[i-1, i:] with itself, scaled by 1/(m + D[i-1, i-1]), from
    D[i:, i:] (what the accompanying text describes).
  * Algorithm 2 (Appendix B): as printed it divides q twice. The recursion of
    Section 3.2 (multiplication) is followed instead: for each i in order,
    first q_i <- q_i / (m + D_ii), then q_j <- q_j - D_ij q_i for j > i.
  * Algorithm 3 (Appendix C): the first denominator is q_1 = m + v_1^T g_1 as
    in the definition q_j = m + g_j^T v_j (Section 3.1); the printed first line
    omits the "m +".
  * Appendix C row-selected extraction: the sum runs over i with 1/q_i.
"""

import numpy as np


# --------------------------------------------------------------------------
# Static algorithm (Section 3.1, eq. 3-5; Appendix C eq. 9 and Algorithm 3)
# --------------------------------------------------------------------------

def static_precompute(G, lam, m=None):
    """V (m x d) and q (m): v_i = F_{i-1}^-1 g_i, q_i = m + g_i^T v_i.

    F_{i-1}^-1 g is evaluated with the unrolled recursion over the already
    computed v_1..v_{i-1} (eq. 4), i.e. Algorithm 3's row step
    v_i = g_i / lambda - sum_{j<i} v_j (v_j^T g_i) / q_j.
    """
    G = np.asarray(G, dtype=np.float64)
    mm = G.shape[0] if m is None else m
    V = np.empty_like(G)
    q = np.empty(G.shape[0])
    for i in range(G.shape[0]):
        g = G[i]
        if i == 0:
            v = g / lam
        else:
            coef = (V[:i] @ g) / q[:i]
            v = g / lam - coef @ V[:i]
        V[i] = v
        q[i] = mm + v @ g
    return V, q


def static_ihvp(V, q, lam, x):
    """F^-1 x = x / lambda - V^T ((V x) / q)  (Appendix C eq. 9)."""
    x = np.asarray(x, dtype=np.float64)
    return x / lam - V.T @ ((V @ x) / q)


def static_element(V, q, lam, i, j):
    """[F^-1]_ij = delta_ij / lambda - sum_k V[k, i] V[k, j] / q_k  (eq. 5)."""
    return (1.0 / lam if i == j else 0.0) - np.sum(V[:, i] * V[:, j] / q)


def static_inv_diag(V, q, lam):
    """diag(F^-1) = 1/lambda - sum_i v_i (.) v_i / q_i  (Appendix C, pi = id)."""
    return 1.0 / lam - np.sum(V * V / q[:, None], axis=0)


# --------------------------------------------------------------------------
# Dynamic algorithm (Section 3.2, eq. 6-8, Theorem 1; Appendix B Alg. 1-2)
# --------------------------------------------------------------------------

def dynamic_D(GG, lam, m):
    """Upper-triangular D with D_ij = g_i^T F_{i-1}^-1 g_j for i <= j.

    Start from D = GG / lambda (that is g_j^T F_0^-1 g_k). Row i is final once
    all earlier rows have been folded in; folding row i-1 into the trailing
    block is the Sherman-Morrison step of Section 3.2 written for scalar
    products (Algorithm 1, first loop).
    """
    D = np.array(GG, dtype=np.float64) / lam
    n = D.shape[0]
    for i in range(1, n):
        r = D[i - 1, i:]
        D[i:, i:] -= np.outer(r, r) / (m + D[i - 1, i - 1])
    return np.triu(D)


def dynamic_B(D, lam, m):
    """Lower-triangular B, B_ii = 1/lambda, B_ij = -sum_{k=j}^{i-1} D_ki/(m+D_kk) B_kj.

    eq. 7, filled row by row (Algorithm 1, second loop): row i is a negative
    combination of the earlier rows with weights D[:i, i] / (m + diag(D)[:i]).
    """
    n = D.shape[0]
    B = np.eye(n) / lam
    piv = m + np.diag(D)
    for i in range(1, n):
        w = -D[:i, i] / piv[:i]
        B[i, :i] = w @ B[:i, :i]
    return B


def dynamic_q(D, p, lam, m):
    """q_i = (g_i^T F_{i-1}^-1 x) / (m + D_ii) from p = G x (Section 3.2).

    Running values start at g_j^T F_0^-1 x = p_j / lambda; after q_i is known,
    every later running value loses D_ij * q_i.
    """
    q = np.asarray(p, dtype=np.float64) / lam
    q = q.copy()
    n = q.shape[0]
    for i in range(n):
        q[i] /= (m + D[i, i])
        q[i + 1:] -= q[i] * D[i, i + 1:]
    return q


def dynamic_ihvp(G, D, B, lam, m, x):
    """F^-1 x = x/lambda - sum_j (sum_{k>=j} q_k B_kj) g_j  (eq. 8)."""
    G = np.asarray(G, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    q = dynamic_q(D, G @ x, lam, m)
    c = B.T @ q
    return x / lam - G.T @ c


def dynamic_coefficients(D, B, p, lam, m):
    """c_j = sum_{k>=j} q_k B_kj (Theorem 1 with i = m)."""
    return B.T @ dynamic_q(D, p, lam, m)
