"""Pins of the dynamic (sliding-window) oracle against things other than itself.

Each test names what fixes the expected value: a hand-derived case, the dense
d x d solve, a closed form, an invariant, or the paper's D/B/q recursion
(Theorem 1, Section 3.2). A dropped term, a wrong sign, a transposed operand or
a wrong 1/m scale in oracle/dynamic.py fails at least one of them.
"""

import numpy as np
import pytest
import scipy.linalg as sla

from oracle import bruteforce, recursions
from oracle.dynamic import WindowOracle


def _rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def _rand_window(rng, m, d, scale=1.0):
    return (rng.standard_normal((m, d)) * scale / np.sqrt(d)).astype(np.float32)


@pytest.mark.parametrize("name", ["sherman_morrison_m1_d2", "orthogonal_rows_m2_d2", "coupled_m2_d3"])
def test_handworked_values(golden, name):
    c = golden[name]
    G = np.array(c["G"], np.float32)
    o = WindowOracle(G.shape[1], c["m"], c["lam"], G0=G)
    Y = o.ihvp(np.array(c["X"], np.float32))
    np.testing.assert_allclose(Y, np.array(c["Y"]), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("m,d,lam", [(1, 7, 0.3), (3, 64, 1e-2), (16, 300, 1e-3), (16, 200, 1e-6), (40, 96, 1e-4)])
def test_matches_dense_solve(m, d, lam):
    """Section 2: the method equals the direct computation with explicit F."""
    rng = np.random.default_rng(m * 1000 + d)
    G = _rand_window(rng, m, d)
    X = rng.standard_normal((3, d)).astype(np.float32)
    o = WindowOracle(d, m, lam, G0=G)
    assert _rel(o.ihvp(X), bruteforce.ihvp(G, lam, X)) < 1e-10
    # the inserted-row query (x is a row of G): the case the optimizer always hits
    assert _rel(o.ihvp(G[1 % m]), bruteforce.ihvp(G, lam, G[1 % m])) < 1e-10


def test_sherman_morrison_m1_closed_form():
    """m = 1: F^-1 x = (x - g (g^T x) / (lambda + |g|^2)) / lambda (Section 2 eq. 2)."""
    rng = np.random.default_rng(1)
    d, lam = 20000, 1e-3
    g = rng.standard_normal(d).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    g64, x64 = g.astype(np.float64), x.astype(np.float64)
    expect = (x64 - g64 * (g64 @ x64) / (lam + g64 @ g64)) / lam
    o = WindowOracle(d, 1, lam, G0=g[None, :])
    assert _rel(o.ihvp(x), expect) < 1e-12


def test_zero_window_is_scaled_identity():
    d, m, lam = 1000, 8, 1e-2
    o = WindowOracle(d, m, lam)
    x = np.random.default_rng(2).standard_normal(d).astype(np.float32)
    np.testing.assert_allclose(o.ihvp(x), x.astype(np.float64) / lam, rtol=0, atol=0)


def test_orthogonal_rows_closed_form():
    """Orthogonal gradients: y = x/lam - sum_i g_i (g_i^T x) / (lam (m lam + |g_i|^2))."""
    rng = np.random.default_rng(3)
    d, m, lam = 4096, 12, 1e-3
    Q, _ = np.linalg.qr(rng.standard_normal((d, m)))
    norms = np.linspace(0.5, 3.0, m)
    # build rows that are exactly orthogonal after fp32 rounding: integer patterns on disjoint supports
    G = np.zeros((m, d), np.float32)
    for i in range(m):
        sl = slice(i * (d // m), (i + 1) * (d // m))
        G[i, sl] = np.sign(Q[sl, i]) * norms[i] / np.sqrt(d // m)
    x = rng.standard_normal(d).astype(np.float32)
    G64, x64 = G.astype(np.float64), x.astype(np.float64)
    expect = x64 / lam
    for i in range(m):
        gi = G64[i]
        expect = expect - gi * (gi @ x64) / (lam * (m * lam + gi @ gi))
    o = WindowOracle(d, m, lam, G0=G)
    assert _rel(o.ihvp(x), expect) < 1e-12


def test_matrix_free_residual_large_d():
    """F y = x checked without forming F: lam y + G^T (G y) / m = x."""
    rng = np.random.default_rng(4)
    d, m, lam = 200_000, 32, 1e-4
    s = np.exp(rng.standard_normal(d))
    G = (rng.standard_normal((m, d)) * s / np.sqrt(d)).astype(np.float32)
    o = WindowOracle(d, m, lam, G0=G)
    for x in (rng.standard_normal(d).astype(np.float32), G[5]):
        y = o.ihvp(x)
        G64 = G.astype(np.float64)
        r = lam * y + G64.T @ (G64 @ y) / m - x.astype(np.float64)
        assert np.linalg.norm(r) / np.linalg.norm(x) < 1e-11


def test_symmetry_positivity_and_bound():
    rng = np.random.default_rng(5)
    d, m, lam = 3000, 20, 1e-3
    G = _rand_window(rng, m, d)
    o = WindowOracle(d, m, lam, G0=G)
    x = rng.standard_normal(d).astype(np.float32)
    z = rng.standard_normal(d).astype(np.float32)
    yx, yz = o.ihvp(x), o.ihvp(z)
    assert abs(z @ yx - yz @ x) <= 1e-11 * abs(z @ yx) + 1e-9
    assert yx @ x > 0
    assert np.linalg.norm(yx) <= np.linalg.norm(x.astype(np.float64)) / lam * (1 + 1e-12)


def test_row_permutation_invariance_and_sliding_equals_fresh():
    """The IHVP depends on the set of rows only; a slid window equals a fresh one."""
    rng = np.random.default_rng(6)
    d, m, lam = 2048, 16, 1e-3
    G0 = _rand_window(rng, m, d)
    o = WindowOracle(d, m, lam, G0=G0)
    news = _rand_window(rng, 23, d)
    ys = [o.slide(g) for g in news]
    fresh = WindowOracle(d, m, lam, G0=o.G.copy())
    perm = np.random.default_rng(7).permutation(m)
    permuted = WindowOracle(d, m, lam, G0=o.G[perm].copy())
    x = rng.standard_normal(d).astype(np.float32)
    assert _rel(o.ihvp(x), fresh.ihvp(x)) < 1e-12
    assert _rel(permuted.ihvp(x), fresh.ihvp(x)) < 1e-11
    # the last slide returned F^-1 g_new for the window holding g_new
    assert _rel(ys[-1], fresh.ihvp(news[-1])) < 1e-12
    # ring order: 23 slides into m = 16 slots, last one went into slot 22 % 16
    np.testing.assert_array_equal(o.G[22 % m], news[-1])
    # incremental Gram equals a fresh one
    assert _rel(o.K, fresh.K) < 1e-13


def test_fill_from_empty_equals_init():
    """An empty window filled by m replaces equals init with those rows."""
    rng = np.random.default_rng(8)
    d, m, lam = 1024, 8, 1e-3
    rows = _rand_window(rng, m, d)
    o = WindowOracle(d, m, lam)
    for g in rows:
        o.slide(g)
    x = rng.standard_normal(d).astype(np.float32)
    assert _rel(o.ihvp(x), WindowOracle(d, m, lam, G0=rows).ihvp(x)) < 1e-12


# ---------------------------------------------------------------------------
# the paper's recursions (oracle/recursions.py) against definitions and O1
# ---------------------------------------------------------------------------

def test_recursions_handworked(golden):
    c = golden["coupled_m2_d3"]
    G = np.array(c["G"], np.float64)
    lam, m = c["lam"], c["m"]
    D = recursions.dynamic_D(G @ G.T, lam, m)
    B = recursions.dynamic_B(D, lam, m)
    np.testing.assert_allclose(D, c["D"], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(B, c["B"], rtol=1e-14, atol=1e-14)
    p = G @ np.array(c["X"][0], np.float64)
    np.testing.assert_allclose(recursions.dynamic_q(D, p, lam, m), c["q"], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(recursions.dynamic_coefficients(D, B, p, lam, m), c["c"], rtol=1e-14, atol=1e-15)


def test_D_and_B_match_their_definitions():
    """D_ij = g_i^T F_{i-1}^-1 g_j (i <= j); F_{k-1}^-1 g_k = sum_j B_kj g_j (Theorem 1)."""
    rng = np.random.default_rng(9)
    d, m, lam = 40, 6, 1e-2
    G = rng.standard_normal((m, d)) / np.sqrt(d)
    D = recursions.dynamic_D(G @ G.T, lam, m)
    B = recursions.dynamic_B(D, lam, m)
    for i in range(m):
        Fi = lam * np.eye(d) + (G[:i].T @ G[:i]) / m   # F_{i-1} in 1-based terms: first i rows
        v = np.linalg.solve(Fi, G[i])
        for j in range(i, m):
            assert abs(D[i, j] - G[j] @ v) < 1e-10 * max(1.0, abs(D[i, j]))
        np.testing.assert_allclose(B[i] @ G, v, rtol=1e-9, atol=1e-9)
        assert np.all(B[i, i + 1:] == 0)


def test_D_equals_scaled_cholesky_factor():
    """D = U(LU_nopivot(K/lam + m I)) - m I (Appendix B), via LAPACK Cholesky R."""
    rng = np.random.default_rng(10)
    d, m, lam = 500, 24, 1e-3
    G = rng.standard_normal((m, d)) / np.sqrt(d)
    K = G @ G.T
    D = recursions.dynamic_D(K, lam, m)
    R = np.linalg.cholesky(K / lam + m * np.eye(m))
    U = np.diag(np.diag(R)) @ R.T
    np.testing.assert_allclose(D, np.triu(U - m * np.eye(m)), rtol=1e-11, atol=1e-9)
    # B = lam^-1 (R diag(R)^-1)^-1, the inverse of the unit lower factor
    Lunit = R / np.diag(R)[None, :]
    B = recursions.dynamic_B(D, lam, m)
    np.testing.assert_allclose(B, np.linalg.inv(Lunit) / lam, rtol=1e-10, atol=1e-8)


def test_combined_update_identity():
    """x = g_i: q_k = D_ki / (m + D_kk) for k <= i (Appendix B, update-multiply)."""
    rng = np.random.default_rng(11)
    d, m, lam = 300, 10, 1e-3
    G = rng.standard_normal((m, d)) / np.sqrt(d)
    D = recursions.dynamic_D(G @ G.T, lam, m)
    for i in range(m):
        q = recursions.dynamic_q(D, G @ G[i], lam, m)
        np.testing.assert_allclose(q[:i + 1], D[:i + 1, i] / (m + np.diag(D)[:i + 1]), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("m,d,lam", [(16, 4096, 1e-3), (64, 2000, 1e-5), (5, 333, 1e-1)])
def test_paper_recursion_equals_woodbury_oracle(m, d, lam):
    """Theorem 1: eq. 8 with D, B, q equals the plain-definition oracle."""
    rng = np.random.default_rng(m + d)
    G = _rand_window(rng, m, d)
    G64 = G.astype(np.float64)
    D = recursions.dynamic_D(G64 @ G64.T, lam, m)
    B = recursions.dynamic_B(D, lam, m)
    o = WindowOracle(d, m, lam, G0=G)
    for x in (rng.standard_normal(d).astype(np.float32), G[m // 2]):
        assert _rel(recursions.dynamic_ihvp(G64, D, B, lam, m, x), o.ihvp(x)) < 1e-10


def test_woodbury_recursion_equals_dense_inverse():
    """Section 2 eq. 2 folded row by row from lambda^-1 I equals inv(F)."""
    rng = np.random.default_rng(12)
    G = rng.standard_normal((7, 30)) / 5.0
    np.testing.assert_allclose(bruteforce.woodbury_recursive_inverse(G, 0.1),
                               np.linalg.inv(bruteforce.fisher(G, 0.1)), rtol=1e-10, atol=1e-10)


def test_oracle_detects_planted_mistakes():
    """The pins above are sharp: plausible slips in the formula move the result."""
    rng = np.random.default_rng(13)
    d, m, lam = 256, 8, 1e-3
    G = _rand_window(rng, m, d)
    x = rng.standard_normal(d).astype(np.float32)
    truth = bruteforce.ihvp(G, lam, x)
    G64, x64 = G.astype(np.float64), x.astype(np.float64)
    K = G64 @ G64.T
    good = (x64 - G64.T @ sla.solve(K + m * lam * np.eye(m), G64 @ x64)) / lam
    assert _rel(good, truth) < 1e-10
    wrong_scale = (x64 - G64.T @ sla.solve(K + lam * np.eye(m), G64 @ x64)) / lam
    wrong_sign = (x64 + G64.T @ sla.solve(K + m * lam * np.eye(m), G64 @ x64)) / lam
    dropped = x64 / lam
    for bad in (wrong_scale, wrong_sign, dropped):
        assert _rel(bad, truth) > 1e-3


def test_gram_accumulate_over_column_ranges_matches_dense_product():
    """The chunk-range Gram that large-window tests use (uneven ranges, chunks
    smaller than a range) equals the fp64 product of the whole matrix, and a
    window built from it gives the dense-solve IHVPs (Section 3.2 initial
    setup: K = G G^T)."""
    from oracle import dynamic as odyn
    rng = np.random.default_rng(31)
    m, d, lam = 9, 1000, 1e-3
    G = _rand_window(rng, m, d)
    K = np.zeros((m, m), np.float64, order="F")
    for j0, j1 in ((0, 333), (333, 334), (334, 901), (901, 1000)):
        K = odyn.gram_accumulate(G, K, j0, j1, chunk=128)
    K = odyn.gram_symmetric(K)
    G64 = G.astype(np.float64)
    assert _rel(K, G64 @ G64.T) < 1e-14
    assert np.array_equal(K, K.T)
    o = WindowOracle(d, m, lam, G0=G, K=K)
    X = rng.standard_normal((2, d)).astype(np.float32)
    assert _rel(o.ihvp(X), bruteforce.ihvp(G, lam, X)) < 1e-10
    # ranges that miss columns give a different matrix (the test would see it)
    K2 = odyn.gram_symmetric(odyn.gram_accumulate(G, np.zeros((m, m), order="F"), 0, 999, chunk=128))
    assert _rel(K2, G64 @ G64.T) > 1e-6
