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
