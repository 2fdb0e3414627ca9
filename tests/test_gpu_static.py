"""GPU parity of the static block-wise path: inverse diagonal, W, scores, mask."""

import os

import numpy as np
import pytest
import scipy.linalg as sla
import torch

from gpu_common import rel_l2, require_gpu, say
from oracle import mask as omask
from oracle import static as ostatic
from synth import GradientStream, get_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _oracle_W(G, lam, B):
    """W_b = R_b^-1 G_b per block (fp64), the quantity written over G."""
    m, d = G.shape
    out = np.empty((m, d))
    for b in range(d // B):
        Gb = G[:, b * B:(b + 1) * B].astype(np.float64)
        R = np.linalg.cholesky(Gb @ Gb.T + m * lam * np.eye(m))
        out[:, b * B:(b + 1) * B] = sla.solve_triangular(R, Gb, lower=True)
    return out


def _run(dev, G, B, lam, theta, keep):
    from paper_2107_03356_amd import StaticBlocks
    Gd = G.to(dev).contiguous()
    sb = StaticBlocks(Gd, B, lam)
    diag64 = sb.inv_diag(fp64=True)
    diag32 = sb.inv_diag()
    mask, scores = sb.obs_mask(theta.to(dev), keep)
    torch.cuda.synchronize()
    assert sb.status() == 0
    return (Gd.cpu().numpy(), diag64.cpu().numpy(), diag32.cpu().numpy(), mask.cpu().numpy(),
            scores.cpu().numpy())


@pytest.mark.parametrize("m,B,nb,lam,batch_cap", [
    (100, 256, 6, 1e-3, None),     # m padded to 128 inside
    (64, 512, 3, 1e-4, 2),         # batch boundary inside the block loop
    (1, 64, 4, 1e-2, None),        # m = 1 closed form
    (200, 2048, 2, 1e-4, None),    # the pruning block width
    (300, 512, 3, 1e-4, None),     # padded to 320: uneven splits in the recursive factor
    (700, 2048, 2, 1e-4, None),    # padded to 704: 11 tiles, half tiles at several levels
    (1500, 512, 3, 1e-4, None),    # m > B and m > 1024: rank-deficient Gram, padded to 1536
    (256, 65536, 1, 1e-4, None),   # B = d (full-d precompute): Gram columns split over 32 work-groups
    (100, 20000, 1, 1e-3, None),   # B = d not a multiple of 32: 9 column splits, ragged last split
    (1024, 16384, 2, 1e-4, None),  # two wide blocks at m = 1024: 8 splits of 36 tiles each
    (64, 8192, 3, 1e-4, 2),        # split Gram in a batch of 2 blocks and a last batch of 1
    (8192, 1024, 2, 1e-3, None),   # the largest m (8192 > B): 2080 Gram tiles, seven recursion levels
])
def test_static_small(dev, m, B, nb, lam, batch_cap, monkeypatch):
    if batch_cap:
        monkeypatch.setenv("MFAC_STATIC_BATCH_BLOCKS", str(batch_cap))
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=B * nb, m=m, block=B, lam=lam, scale_d=B)   # per-block scale: Fisher term well above m*lam
    gs = GradientStream(wl, seed=11)
    G = gs.rows(0, m)
    theta = gs.theta()
    keep = wl.d // 2
    say("static small", m, B, nb, lam, batch_cap)
    W, d64, d32, mk, sc = _run(dev, G, B, lam, theta, keep)
    Gn = G.numpy()
    dref = ostatic.inv_diag(Gn, lam, B)
    assert rel_l2(d64, dref) < 1e-11
    assert rel_l2(d32, dref) < 1e-6
    assert rel_l2(W, _oracle_W(Gn, lam, B)) < 1e-6
    sref = omask.scores(theta.numpy(), dref)
    assert rel_l2(sc, sref) < 1e-11
    np.testing.assert_array_equal(mk, omask.keep_mask(sref, keep))


def test_static_pruning_recipe_reduced_blocks(dev):
    """m = 1024, B = 2048 with the full-size entry scale (1/sqrt(4,194,304)), 3 blocks."""
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=3 * 2048, scale_d=base.d)
    gs = GradientStream(wl, seed=0)
    G = gs.rows(0, wl.m)
    theta = gs.theta()
    keep = wl.d // 2
    say("static pruning recipe, 3 blocks")
    W, d64, d32, mk, sc = _run(dev, G, wl.block, wl.lam, theta, keep)
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block)
    assert rel_l2(d64, dref) < 1e-11
    sref = omask.scores(theta.numpy(), dref)
    np.testing.assert_array_equal(mk, omask.keep_mask(sref, keep))


@pytest.mark.parametrize("keep_frac", [0.0, 1.0, 1e-4, 0.5, 0.7])
def test_mask_edges_and_ties(dev, keep_frac):
    """keep = 0, d, 1, and cuts inside a band of exactly tied (zero) scores."""
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=8 * 256, m=48, block=256, lam=1e-3, scale_d=256)
    gs = GradientStream(wl, seed=12)
    G = gs.rows(0, wl.m)
    theta = gs.theta()
    theta[::3] = 0.0            # a third of the scores are exactly 0: ties at the cut for keep > 2/3 d
    theta[1::7] = -0.0
    keep = int(round(wl.d * keep_frac))
    say("mask edges", keep)
    W, d64, d32, mk, sc = _run(dev, G, wl.block, wl.lam, theta, keep)
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block)
    sref = omask.scores(theta.numpy(), dref)
    np.testing.assert_array_equal(mk, omask.keep_mask(sref, keep))
    assert int(mk.sum()) == keep


@pytest.mark.parametrize("m,B,nb,lam,scale_full", [
    (100, 256, 6, 1e-3, False),
    (1024, 2048, 2, 1e-4, True),     # pruning block width and m, full-size entry scale
    (37, 100, 3, 1e-2, False),       # B not a multiple of the chunk widths, m padded
    (64, 65536, 1, 1e-3, False),     # B = d: 128 pass-1 chunks per block, summed in 2 segments
    (128, 262144, 1, 1e-4, False),   # B = d: segmented chunk sums for 1 and for 3 vectors
])
def test_static_ihvp_element_and_obs_update(dev, m, B, nb, lam, scale_full):
    from paper_2107_03356_amd import StaticBlocks
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=B * nb, m=m, block=B, lam=lam, scale_d=(base.d if scale_full else B))
    gs = GradientStream(wl, seed=31)
    G = gs.rows(0, m)
    theta = gs.theta()
    X = gs.queries(0, 3)
    say("static queries", m, B, nb)
    sb = StaticBlocks(G.to(dev).contiguous(), B, lam)
    Y = sb.ihvp(X.to(dev).contiguous())
    Gn, Xn = G.numpy(), X.numpy()
    Yo = ostatic.ihvp(Gn, lam, B, Xn)
    for q in range(3):
        assert rel_l2(Y[q].cpu().numpy(), Yo[q]) < 1e-4
    # element queries: same block, diagonal, across blocks, ragged positions
    rng = np.random.default_rng(5)
    pairs = [(0, 0), (1, 2), (B - 1, 0), (B, B + 3), (wl.d - 1, wl.d - 2), (3, B + 3), (B // 2, B // 2)]
    pairs += [(int(i), int(i // B * B + rng.integers(0, B))) for i in rng.integers(0, wl.d, 20)]
    pairs = [(i, j) for i, j in pairs if i < wl.d and j < wl.d]    # one block: no second block to pair with
    ij = torch.tensor(pairs, dtype=torch.int64)
    el = sb.element(ij).cpu().numpy()
    ref = np.array([ostatic.element(Gn, lam, B, i, j) for i, j in pairs])
    scale = np.abs(ref).max()
    assert np.max(np.abs(el - ref)) < 1e-5 * scale
    # OBS correction for the complement of the 50% keep-mask
    keep = wl.d // 2
    mask, _ = sb.obs_mask(theta.to(dev), keep)
    delta = sb.obs_update(theta.to(dev), mask)
    torch.cuda.synchronize()
    assert sb.status() == 0
    dref = ostatic.obs_update(Gn, lam, B, theta.numpy(), mask.cpu().numpy())
    assert rel_l2(delta.cpu().numpy(), dref) < 1e-4


def test_obs_single_weight_and_bad_element_index(dev):
    from paper_2107_03356_amd import MFAC_ENONFINITE, StaticBlocks
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=4 * 512, m=64, block=512, lam=1e-3, scale_d=512)
    gs = GradientStream(wl, seed=32)
    G = gs.rows(0, wl.m)
    theta = gs.theta()
    say("obs single weight")
    sb = StaticBlocks(G.to(dev).contiguous(), wl.block, wl.lam)
    mask = torch.ones(wl.d, dtype=torch.uint8)
    mask[700] = 0
    delta = sb.obs_update(theta.to(dev), mask.to(dev)).cpu().numpy()
    th = theta.numpy().astype(np.float64)
    assert abs(th[700] + delta[700]) < 1e-4 * abs(th[700])     # the removed weight goes to zero
    assert np.all(delta[:512] == 0) and np.all(delta[1024:] == 0)  # only its block moves
    out = sb.element(torch.tensor([[0, wl.d]], dtype=torch.int64)).cpu().numpy()
    assert np.isnan(out[0])
    assert sb.status() == MFAC_ENONFINITE
    assert sb.status() == 0


def test_nonfinite_gradient_latches_and_other_blocks_stay_exact(dev):
    """A NaN in one block of G latches MFAC_ENONFINITE (its pivots are not
    positive); blocks are independent, so the other blocks' diagonals still
    match the oracle."""
    from paper_2107_03356_amd import MFAC_ENONFINITE, StaticBlocks
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=3 * 256, m=40, block=256, lam=1e-3, scale_d=256)
    gs = GradientStream(wl, seed=41)
    G = gs.rows(0, wl.m)
    Gbad = G.clone()
    Gbad[7, 256 + 13] = float("nan")
    say("static nonfinite")
    sb = StaticBlocks(Gbad.to(dev).contiguous(), wl.block, wl.lam)
    d64 = sb.inv_diag(fp64=True).cpu().numpy()
    assert sb.status() == MFAC_ENONFINITE
    assert sb.status() == 0                      # the latch clears once reported
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block, blocks=[0, 2])
    got = np.concatenate([d64[:256], d64[512:]])
    assert rel_l2(got, dref) < 1e-11


def test_many_element_queries(dev):
    """300,000 element queries (more than one query per wave of the capped
    grid) against dense per-block inverses."""
    from paper_2107_03356_amd import StaticBlocks
    from oracle import bruteforce
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=4 * 256, m=16, block=256, lam=1e-3, scale_d=256)
    gs = GradientStream(wl, seed=44)
    G = gs.rows(0, wl.m)
    say("static many element queries")
    sb = StaticBlocks(G.to(dev).contiguous(), wl.block, wl.lam)
    rng = np.random.default_rng(8)
    nq = 300_000
    i = rng.integers(0, wl.d, nq)
    same = rng.random(nq) < 0.8
    j = np.where(same, i // wl.block * wl.block + rng.integers(0, wl.block, nq), rng.integers(0, wl.d, nq))
    ij = torch.tensor(np.stack([i, j], axis=1), dtype=torch.int64)
    el = sb.element(ij).cpu().numpy()
    assert sb.status() == 0
    Gn = G.numpy()
    inv = [np.linalg.inv(bruteforce.fisher(Gn[:, b * wl.block:(b + 1) * wl.block], wl.lam, wl.m))
           for b in range(wl.d // wl.block)]
    bi, bj = i // wl.block, j // wl.block
    ref = np.zeros(nq)
    for b in range(wl.d // wl.block):
        sel = (bi == b) & (bj == b)
        ref[sel] = inv[b][i[sel] - b * wl.block, j[sel] - b * wl.block]
    assert np.max(np.abs(el - ref)) < 1e-5 * np.abs(ref).max()
    assert np.all(el[bi != bj] == 0.0)


def test_nonfinite_theta_latches_and_mask_keeps_its_count(dev):
    """Non-finite weights latch MFAC_ENONFINITE from the score stage; the mask
    still keeps exactly `keep` coordinates, and the finite coordinates' scores
    match the oracle."""
    from paper_2107_03356_amd import MFAC_ENONFINITE, StaticBlocks
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=4 * 256, m=32, block=256, lam=1e-3, scale_d=256)
    gs = GradientStream(wl, seed=43)
    G = gs.rows(0, wl.m)
    theta = gs.theta()
    theta[5] = float("nan")
    theta[300] = float("inf")
    theta[301] = float("-inf")
    say("static nonfinite theta")
    sb = StaticBlocks(G.to(dev).contiguous(), wl.block, wl.lam)
    assert sb.status() == 0
    keep = wl.d // 2
    mask, sc = sb.obs_mask(theta.to(dev), keep)
    mk, sc = mask.cpu().numpy(), sc.cpu().numpy()
    assert sb.status() == MFAC_ENONFINITE
    assert sb.status() == 0
    assert int(mk.sum()) == keep
    fin = np.isfinite(theta.numpy())
    sref = omask.scores(theta.numpy(), ostatic.inv_diag(G.numpy(), wl.lam, wl.block))
    assert rel_l2(sc[fin], sref[fin]) < 1e-11


def test_stage_trace_counts_and_unchanged_results(dev, monkeypatch):
    """MFAC_STATIC_TRACE: one interval per batch for the Gram, factor and W
    stages and one per mask call; tracing leaves every output bit-identical."""
    from paper_2107_03356_amd import StaticBlocks
    monkeypatch.setenv("MFAC_STATIC_BATCH_BLOCKS", "2")
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=5 * 512, m=96, block=512, lam=1e-3, scale_d=512)
    gs = GradientStream(wl, seed=13)
    G = gs.rows(0, wl.m)
    theta = gs.theta().to(dev)
    say("static trace", wl.d, wl.m)
    outs = []
    for trace in (False, True):
        sb = StaticBlocks(G.to(dev).contiguous(), wl.block, wl.lam, trace=trace)
        d64 = sb.inv_diag(fp64=True)
        mask, sc = sb.obs_mask(theta, wl.d // 2)
        torch.cuda.synchronize()
        assert sb.status() == 0
        ms, cnt = sb.trace_read()
        outs.append((d64.cpu().numpy(), mask.cpu().numpy(), sc.cpu().numpy(), list(ms), list(cnt)))
        sb.close()
    (d0, m0, s0, ms0, c0), (d1, m1, s1, ms1, c1) = outs
    np.testing.assert_array_equal(d0, d1)
    np.testing.assert_array_equal(m0, m1)
    np.testing.assert_array_equal(s0, s1)
    assert c0 == [0, 0, 0, 0] and ms0 == [0.0] * 4
    assert c1 == [3, 3, 3, 1]                  # 5 blocks in batches of 2, 2, 1; one mask call
    assert all(t > 0.0 for t in ms1)
