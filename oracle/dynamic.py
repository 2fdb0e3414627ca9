"""Sliding-window IHVP oracle: y = F^-1 x in float64 (test infrastructure only).

Definition followed (Theorem 1, Section 3.2; sliding window of Section 4.2):
    F = lambda * I_d + (1/m) * G^T G,   G = the m x d window, one gradient per row.
The 1/m scale is the window capacity m, also while some slots still hold zero
rows (a zero row adds nothing to F).

Evaluation: the Woodbury identity (the closed form that the Sherman-Morrison
recursion of Section 2 eq. 2 unrolls to)
    F^-1 x = (x - G^T (G G^T + m*lambda*I)^-1 G x) / lambda,
with K = G G^T accumulated in float64 from the exact fp32 rows, one LAPACK
Cholesky of K + m*lambda*I and two triangular solves. The paper states the
method is numerically equivalent to the direct computation (Section 2), so the
plain definition is the oracle. Pinned in tests/test_oracle_dynamic.py against
the dense d x d solve, the m = 1 Sherman-Morrison closed form, orthogonal rows,
G = 0, the matrix-free residual F y = x, and the paper's D/B/q recursion.
"""

import numpy as np
import scipy.linalg as sla
import torch

_CHUNK = 1 << 18  # columns per fp64 chunk (bounds the fp64 temporaries)


def _chunks(d, chunk=_CHUNK):
    for j0 in range(0, d, chunk):
        yield j0, min(d, j0 + chunk)


class _F64Chunks:
    """Column chunks of an fp32 matrix converted to float64 in one reused buffer.

    The conversion is exact (every fp32 value is a float64 value); torch's
    CPU copy does it with all threads and without fresh page faults.
    """

    def __init__(self, rows, chunk=_CHUNK, cols=None):
        # the buffer is as wide as one chunk, or as the matrix when it is narrower
        width = chunk if cols is None else max(1, min(chunk, cols))
        self.buf = np.empty((rows, width), np.float64)
        self.chunk = chunk

    def __call__(self, A):
        d = A.shape[1]
        for j0, j1 in _chunks(d, self.chunk):
            b = self.buf[:A.shape[0], :j1 - j0]
            torch.from_numpy(b).copy_(torch.from_numpy(A[:, j0:j1]))
            yield j0, j1, b


def gram_accumulate(G, K, j0, j1, chunk=_CHUNK):
    """Add the lower triangle of G[:, j0:j1] G[:, j0:j1]^T to K in float64.

    K is an m x m float64 array in Fortran order (start from zeros). Each
    column chunk's product is the BLAS symmetric rank-k update (dsyrk) of the
    chunk converted to float64; only the lower triangle of K is formed.
    Calling it over consecutive column ranges that cover [0, d) and then
    ``gram_symmetric`` gives ``gram(G)``; the returned K must be passed on
    (dsyrk may return a new array).
    """
    m = G.shape[0]
    conv = _F64Chunks(m, chunk, j1 - j0)
    for a in range(j0, j1, chunk):
        b = conv.buf[:, :min(j1, a + chunk) - a]
        torch.from_numpy(b).copy_(torch.from_numpy(G[:, a:a + b.shape[1]]))
        K = sla.blas.dsyrk(1.0, b.T, beta=1.0, c=K, trans=1, lower=1, overwrite_c=1)
    return K


def gram_symmetric(K):
    """The full symmetric Gram matrix (C order) from its accumulated lower triangle."""
    L = np.tril(K)
    return np.ascontiguousarray(L + np.tril(L, -1).T)


def gram(G, chunk=_CHUNK):
    """K = G G^T in float64 from fp32 rows, accumulated over column chunks
    (``gram_accumulate`` over all d columns, then mirrored)."""
    m, d = G.shape
    K = np.zeros((m, m), np.float64, order="F")
    return gram_symmetric(gram_accumulate(G, K, 0, d, chunk))


def matvec(G, X, chunk=_CHUNK):
    """P = G X^T (m x n) in float64; X is (n, d) fp32."""
    m, d = G.shape
    P = np.zeros((m, X.shape[0]), np.float64)
    conv = _F64Chunks(m, chunk, d)
    for j0, j1, b in conv(G):
        P += b @ X[:, j0:j1].astype(np.float64).T
    return P


class WindowOracle:
    """The m x d window, its float64 Gram matrix, and exact IHVPs.

    ``G0`` (m x d fp32) initialises the window; None starts with zero rows.
    ``copy=False`` keeps the caller's G0 array as the window (it is then
    modified in place by replace).
    """

    def __init__(self, d, m, lam, G0=None, K=None, copy=True):
        self.d, self.m, self.lam = int(d), int(m), float(lam)
        if G0 is None:
            self.G = np.zeros((m, d), np.float32)
            self.K = np.zeros((m, m), np.float64)
        else:
            self.G = np.array(G0, dtype=np.float32, copy=True) if copy else G0
            assert self.G.shape == (m, d) and self.G.dtype == np.float32
            # K: the Gram matrix of G0 when the caller formed it already (with
            # gram_accumulate over column ranges, for windows too large to
            # redo); otherwise computed here
            self.K = gram(self.G) if K is None else np.array(K, dtype=np.float64)
            assert self.K.shape == (m, m)
        self.steps = 0

    def replace(self, slot, g):
        """Overwrite row ``slot`` with g and refresh row and column slot of K.

        Section 3.2 (initial precomputation and update): only the scalar
        products of the new gradient with the window change.
        """
        g = np.asarray(g, dtype=np.float32)
        self.G[slot] = g
        p = matvec(self.G, g[None, :])[:, 0]
        self.K[slot, :] = p
        self.K[:, slot] = p
        self.steps += 1
        return p

    def slide(self, g):
        """Ring semantics: replace the oldest slot (steps mod m), return F^-1 g.

        Section 4.2: the window drops its oldest gradient, takes the newest, and
        the same newest gradient is then preconditioned. G g after the insert is
        the Gram column the replace just computed (Appendix B reuses it the same
        way), so it is passed on instead of being recomputed.
        """
        slot = self.steps % self.m
        p = self.replace(slot, g)
        return self.ihvp(np.asarray(g, np.float32)[None, :], P=p[:, None])[0]

    def coefficients(self, P):
        """U = (K + m*lambda*I)^-1 P for P (m x n)."""
        A = self.K + self.m * self.lam * np.eye(self.m)
        c, low = sla.cho_factor(A, lower=True)
        return sla.cho_solve((c, low), P)

    def ihvp(self, X, P=None):
        """F^-1 X for X of shape (d,) or (n, d); returns float64 of that shape.

        P = G X^T may be passed when already known.
        """
        X = np.asarray(X, dtype=np.float32)
        single = X.ndim == 1
        if single:
            X = X[None, :]
        if P is None:
            P = matvec(self.G, X)
        U = self.coefficients(P)
        Y = np.empty(X.shape, np.float64)
        for j0, j1, b in _F64Chunks(self.m, cols=self.d)(self.G):
            Y[:, j0:j1] = (X[:, j0:j1].astype(np.float64) - U.T @ b) / self.lam
        return Y[0] if single else Y
