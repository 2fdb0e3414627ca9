"""Pins of the static block-wise inverse-diagonal oracle and the OBD mask."""

import numpy as np
import pytest

from oracle import bruteforce, mask, recursions
from oracle import static as st
from oracle.dynamic import WindowOracle


def _rel(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / np.linalg.norm(np.asarray(b))


@pytest.mark.parametrize("name", ["sherman_morrison_m1_d2", "orthogonal_rows_m2_d2", "coupled_m2_d3"])
def test_handworked_diag(golden, name):
    c = golden[name]
    G = np.array(c["G"], np.float32)
    np.testing.assert_allclose(st.block_inv_diag(G, c["lam"], c["m"]), c["diag"], rtol=1e-13)


@pytest.mark.parametrize("m,B,lam", [(1, 9, 0.5), (4, 64, 1e-2), (32, 128, 1e-4), (64, 48, 1e-3)])
def test_block_diag_matches_dense_inverse(m, B, lam):
    """diag(F_b^-1) from inv(F_b) formed densely (B x B)."""
    rng = np.random.default_rng(m * 7 + B)
    G = (rng.standard_normal((m, B)) / np.sqrt(B)).astype(np.float32)
    assert _rel(st.block_inv_diag(G, lam), bruteforce.inv_diag(G, lam)) < 1e-11


def test_m1_closed_form():
    """m = 1: [F^-1]_jj = (1 - g_j^2 / (m lam + |g|^2)) / lam."""
    rng = np.random.default_rng(1)
    g = rng.standard_normal(5000).astype(np.float32)
    lam = 1e-2
    g64 = g.astype(np.float64)
    expect = (1 - g64 ** 2 / (lam + g64 @ g64)) / lam
    assert _rel(st.block_inv_diag(g[None, :], lam), expect) < 1e-12


def test_trace_identity_and_bounds():
    """sum_j (1/lam - diag_j) = (1/lam) sum_i mu_i / (mu_i + m lam), mu = eig(G_b G_b^T)."""
    rng = np.random.default_rng(2)
    m, B, lam = 48, 256, 1e-3
    s = np.exp(rng.standard_normal(B))
    G = (rng.standard_normal((m, B)) * s / np.sqrt(B)).astype(np.float32)
    dg = st.block_inv_diag(G, lam)
    G64 = G.astype(np.float64)
    mu = np.linalg.eigvalsh(G64 @ G64.T)
    lhs = np.sum(1 / lam - dg)
    rhs = np.sum(mu / (mu + m * lam)) / lam
    assert abs(lhs - rhs) / rhs < 1e-11
    assert np.all(lam * dg > 0) and np.all(lam * dg <= 1 + 1e-12)


def test_small_damping_limit_is_projection():
    """m lam -> 0: lam [F^-1]_jj -> 1 - |P e_j|^2, P the projector on span(rows) (Appendix, normalisation effects)."""
    rng = np.random.default_rng(3)
    m, B = 6, 40
    G = rng.standard_normal((m, B)).astype(np.float32)
    Q, _ = np.linalg.qr(G.astype(np.float64).T)      # B x m orthonormal basis of the row span
    expect = 1 - np.sum(Q * Q, axis=1)
    lam = 1e-9
    got = lam * st.block_inv_diag(G, lam)
    assert np.max(np.abs(got - expect)) < 1e-6


def test_paper_static_algorithm_equals_oracle():
    """Algorithm 3 (V, q) with eq. 9 and the diagonal extraction equals the oracle."""
    rng = np.random.default_rng(4)
    m, B, lam = 20, 150, 1e-3
    G = (rng.standard_normal((m, B)) / np.sqrt(B)).astype(np.float32)
    V, q = recursions.static_precompute(G, lam)
    assert _rel(recursions.static_inv_diag(V, q, lam), st.block_inv_diag(G, lam)) < 1e-11
    x = rng.standard_normal(B)
    assert _rel(recursions.static_ihvp(V, q, lam, x), bruteforce.ihvp(G, lam, x)) < 1e-11
    Finv = np.linalg.inv(bruteforce.fisher(G, lam))
    for (i, j) in [(0, 0), (3, 7), (149, 2), (10, 10)]:
        assert abs(recursions.static_element(V, q, lam, i, j) - Finv[i, j]) < 1e-9 * np.abs(Finv).max()
    # the same block through the dynamic oracle's IHVP
    o = WindowOracle(B, m, lam, G0=G)
    assert _rel(o.ihvp(x.astype(np.float32)), bruteforce.ihvp(G, lam, x.astype(np.float32))) < 1e-10


def test_static_dynamic_link():
    """V = B G and q_i = m + D_ii (Sections 3.1-3.2 share v_i = F_{i-1}^-1 g_i)."""
    rng = np.random.default_rng(5)
    m, d, lam = 12, 90, 1e-2
    G = rng.standard_normal((m, d)) / np.sqrt(d)
    V, q = recursions.static_precompute(G, lam)
    D = recursions.dynamic_D(G @ G.T, lam, m)
    Bm = recursions.dynamic_B(D, lam, m)
    np.testing.assert_allclose(V, Bm @ G, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(q, m + np.diag(D), rtol=1e-12)


def test_blocks_are_independent_and_concatenate():
    rng = np.random.default_rng(6)
    m, B, nb, lam = 8, 32, 5, 1e-3
    G = (rng.standard_normal((m, B * nb)) / np.sqrt(B)).astype(np.float32)
    full = st.inv_diag(G, lam, B)
    for b in range(nb):
        np.testing.assert_array_equal(full[b * B:(b + 1) * B], st.block_inv_diag(G[:, b * B:(b + 1) * B], lam))
    G2 = G.copy()
    G2[:, 2 * B:3 * B] *= 3.0
    full2 = st.inv_diag(G2, lam, B)
    np.testing.assert_array_equal(full[:2 * B], full2[:2 * B])
    assert not np.allclose(full[2 * B:3 * B], full2[2 * B:3 * B])
    np.testing.assert_array_equal(st.inv_diag(G, lam, B, blocks=[3, 1]),
                                  np.concatenate([full[3 * B:4 * B], full[B:2 * B]]))


# ---------------------------------------------------------------------------
# OBD saliency and the global keep-mask
# ---------------------------------------------------------------------------

def test_mask_handworked(golden):
    c = golden["obd_mask_small"]
    s = mask.scores(c["theta"], c["diag_in"])
    np.testing.assert_allclose(s, c["scores"], rtol=1e-15)
    np.testing.assert_array_equal(mask.keep_mask(s, c["keep"]), c["mask"])
    np.testing.assert_array_equal(mask.keep_mask(c["tie_scores"], c["tie_keep"]), c["tie_mask"])


def test_mask_matches_python_sort_with_ties():
    rng = np.random.default_rng(7)
    d = 3001
    s = rng.integers(0, 40, d).astype(np.float64) / 7.0   # many exact ties
    for keep in (0, 1, 1500, 3000, 3001):
        order = sorted(range(d), key=lambda j: (-s[j], j))
        expect = np.zeros(d, np.uint8)
        expect[order[:keep]] = 1
        np.testing.assert_array_equal(mask.keep_mask(s, keep), expect)
        assert mask.keep_mask(s, keep).sum() == keep


def test_keep_count():
    assert mask.keep_count(4_194_304, 0.5) == 2_097_152
    assert mask.keep_count(7, 0.5) == 3


# ---------------------------------------------------------------------------
# static queries: IHVP, element, OBS update (Section 3.1 eq. 5, Appendix C eq. 9, Section 4.1)
# ---------------------------------------------------------------------------

def test_static_ihvp_and_element_match_dense_inverse():
    rng = np.random.default_rng(8)
    m, B, nb, lam = 10, 24, 3, 1e-2
    G = (rng.standard_normal((m, B * nb)) / np.sqrt(B)).astype(np.float32)
    X = rng.standard_normal((2, B * nb)).astype(np.float32)
    Y = st.ihvp(G, lam, B, X)
    for b in range(nb):
        sl = slice(b * B, (b + 1) * B)
        Finv = np.linalg.inv(bruteforce.fisher(G[:, sl], lam))
        np.testing.assert_allclose(Y[:, sl], X[:, sl].astype(np.float64) @ Finv.T, rtol=1e-10, atol=1e-10)
        for (i, j) in [(0, 0), (3, 17), (23, 5)]:
            assert abs(st.element(G, lam, B, b * B + i, b * B + j) - Finv[i, j]) < 1e-9 * np.abs(Finv).max()
    assert st.element(G, lam, B, 1, B + 1) == 0.0          # different blocks
    np.testing.assert_allclose([st.element(G, lam, B, j, j) for j in range(B * nb)], st.inv_diag(G, lam, B),
                               rtol=1e-11)


def test_static_ihvp_equals_paper_eq9():
    """Appendix C eq. 9 with the paper's V and q gives the same block IHVP."""
    rng = np.random.default_rng(9)
    m, B, lam = 16, 64, 1e-3
    G = (rng.standard_normal((m, B)) / np.sqrt(B)).astype(np.float32)
    x = rng.standard_normal(B)
    V, q = recursions.static_precompute(G, lam)
    assert _rel(st.block_ihvp(G, lam, x), recursions.static_ihvp(V, q, lam, x)) < 1e-11


def test_obs_single_weight_zeroes_it():
    """Section 4.1: the OBS correction for one weight sets that weight to zero."""
    rng = np.random.default_rng(10)
    m, B, nb, lam = 8, 32, 2, 1e-2
    G = (rng.standard_normal((m, B * nb)) / np.sqrt(B)).astype(np.float32)
    theta = rng.standard_normal(B * nb) * 0.05
    for i in (3, B + 7):
        keep = np.ones(B * nb, np.uint8)
        keep[i] = 0
        delta = st.obs_update(G, lam, B, theta, keep)
        assert abs(theta[i] + delta[i]) < 1e-12
        # only i's block moves (block-diagonal F)
        other = slice(0, B) if i >= B else slice(B, 2 * B)
        assert np.all(delta[other] == 0)
        # equals -theta_i F^-1 e_i / [F^-1]_ii from the dense inverse
        b = i // B
        Finv = np.linalg.inv(bruteforce.fisher(G[:, b * B:(b + 1) * B], lam))
        li = i - b * B
        np.testing.assert_allclose(delta[b * B:(b + 1) * B], -theta[i] * Finv[:, li] / Finv[li, li],
                                   rtol=1e-9, atol=1e-12)


def test_obs_set_is_sum_of_single_updates():
    rng = np.random.default_rng(11)
    m, B, lam = 6, 20, 1e-2
    G = (rng.standard_normal((m, B)) / np.sqrt(B)).astype(np.float32)
    theta = rng.standard_normal(B) * 0.05
    keep = np.ones(B, np.uint8)
    keep[[2, 9, 13]] = 0
    total = st.obs_update(G, lam, B, theta, keep)
    parts = []
    for i in (2, 9, 13):
        k1 = np.ones(B, np.uint8)
        k1[i] = 0
        parts.append(st.obs_update(G, lam, B, theta, k1))
    np.testing.assert_allclose(total, np.sum(parts, axis=0), rtol=1e-10, atol=1e-13)
