"""Block-wise inverse diagonal of the damped empirical Fisher (test infrastructure only).

Definition followed (Section 3.1, block-wise paragraph; Appendix C, diagonal
extraction): the d coordinates are split into d/B contiguous blocks; block b
has its own
    F_b = lambda * I_B + (1/m) * G_b^T G_b,   G_b = G[:, bB:(b+1)B]  (m x B),
and the query is diag(F_b^-1) for every block.

Evaluation in float64 per block, through the Woodbury identity:
    diag(F_b^-1)_j = (1 - g_j^T (K_b + m*lambda*I)^-1 g_j) / lambda,
with K_b = G_b G_b^T and g_j the j-th column of G_b; using the Cholesky
factor R of K_b + m*lambda*I this is (1 - ||R^-1 g_j||^2) / lambda.
Pinned in tests/test_oracle_static.py against inv(F_b) formed densely, the
m = 1 closed form, the trace identity over eig(K_b), the bound
0 < lambda * diag <= 1, and the paper's V/q recursion (Algorithm 3).
"""

import numpy as np
import scipy.linalg as sla


def block_inv_diag(Gb, lam, m=None):
    """diag(F_b^-1) for one block; Gb is m x B (fp32 values)."""
    Gb = np.asarray(Gb, dtype=np.float64)
    mm = Gb.shape[0] if m is None else m
    K = Gb @ Gb.T
    R = np.linalg.cholesky(K + mm * lam * np.eye(Gb.shape[0]))
    W = sla.solve_triangular(R, Gb, lower=True)
    return (1.0 - np.sum(W * W, axis=0)) / lam


def inv_diag(G, lam, block, blocks=None):
    """diag(F^-1) for the block-wise Fisher over all d coordinates.

    ``blocks`` optionally restricts the work to a list of block indices; the
    returned array then holds only those blocks, concatenated in that order.
    """
    G = np.asarray(G, dtype=np.float32)
    m, d = G.shape
    assert d % block == 0
    nb = d // block
    idx = range(nb) if blocks is None else blocks
    out = []
    for b in idx:
        out.append(block_inv_diag(G[:, b * block:(b + 1) * block], lam, m))
    return np.concatenate(out) if out else np.zeros(0)


def block_ihvp(Gb, lam, X, m=None):
    """F_b^-1 X for one block (X: (n, B) or (B,)), Woodbury in float64:
    (X - G_b^T (G_b G_b^T + m*lambda*I)^-1 G_b X) / lambda.
    """
    Gb = np.asarray(Gb, dtype=np.float64)
    mm = Gb.shape[0] if m is None else m
    X = np.asarray(X, dtype=np.float64)
    single = X.ndim == 1
    if single:
        X = X[None, :]
    A = Gb @ Gb.T + mm * lam * np.eye(Gb.shape[0])
    U = np.linalg.solve(A, Gb @ X.T)
    Y = (X - (Gb.T @ U).T) / lam
    return Y[0] if single else Y


def ihvp(G, lam, block, X):
    """F^-1 X for the block-wise Fisher (block-diagonal F), X: (n, d) or (d,).

    X is used at its own precision (fp32 inputs, or an fp64 vector built by
    obs_update)."""
    G = np.asarray(G, dtype=np.float32)
    m, d = G.shape
    X = np.asarray(X)
    single = X.ndim == 1
    if single:
        X = X[None, :]
    Y = np.empty(X.shape, np.float64)
    for b in range(d // block):
        sl = slice(b * block, (b + 1) * block)
        Y[:, sl] = block_ihvp(G[:, sl], lam, X[:, sl], m)
    return Y[0] if single else Y


def element(G, lam, block, i, j):
    """[F^-1]_ij for the block-wise Fisher: 0 across blocks; within a block the
    (i, j) entry of (I - G_b^T (G_b G_b^T + m*lambda*I)^-1 G_b) / lambda."""
    if i // block != j // block:
        return 0.0
    b = i // block
    Gb = np.asarray(G[:, b * block:(b + 1) * block], dtype=np.float64)
    m = Gb.shape[0]
    A = Gb @ Gb.T + m * lam * np.eye(m)
    gi, gj = Gb[:, i - b * block], Gb[:, j - b * block]
    return ((1.0 if i == j else 0.0) - gi @ np.linalg.solve(A, gj)) / lam


def obs_update(G, lam, block, theta, keep_mask):
    """OBS correction for removing every weight outside the keep-mask at once.

    Section 4.1: removing weight i moves the others by -theta_i F^-1 e_i / [F^-1]_ii;
    for a set of weights the single-weight corrections are summed (the
    approximate simultaneous OBS the paper compares in its appendix):
    delta = -F^-1 x, x_i = theta_i / [F^-1]_ii on removed coordinates, 0 elsewhere.
    """
    theta = np.asarray(theta, dtype=np.float64)
    diag = inv_diag(G, lam, block)
    x = np.where(np.asarray(keep_mask) == 0, theta / diag, 0.0)
    return -ihvp(G, lam, block, x.astype(np.float64))
