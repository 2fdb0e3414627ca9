"""GPU parity of the fast static mode (MFAC_STATIC_FP32) against the fp64 oracle.

The Gram matrices, their factors and W run on fp32 matrix cores; the inverse diagonal then
carries fp32 rounding, while the keep-mask must still equal the oracle's bit
for bit (its band at the cut is recomputed in fp64). Each case checks:
the diagonal and every score against the oracle (the measured score error
far below the band's half-width, 1e-5), the mask bit for bit, G left intact,
and the queries (which form W on first use) against the oracle.
"""

import numpy as np
import pytest
import torch

from gpu_common import REL_TOL, rel_l2, require_gpu, say
from oracle import mask as omask
from oracle import static as ostatic
from synth import GradientStream, get_workload

pytestmark = pytest.mark.gpu

TAU = 1e-5   # the library's band half-width (relative)


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _fast(dev, G, B, lam, theta, keep):
    from paper_2107_03356_amd import StaticBlocks
    Gd = G.to(dev).contiguous()
    sb = StaticBlocks(Gd, B, lam, fp32=True)
    mask, scores = sb.obs_mask(theta.to(dev), keep)
    diag = sb.inv_diag(fp64=True)
    torch.cuda.synchronize()
    st = sb.status()
    return sb, Gd, st, diag.cpu().numpy(), mask.cpu().numpy(), scores.cpu().numpy()


def _certificate(scores, sref, keep):
    """What makes the fast mask exact, measured: every coordinate's score
    error (fp32 path, or fp64 for the band) is well below its relative
    distance to the oracle's cut, or below the band's half-width; near the
    cut the fp32 error is far below that half-width."""
    nz = sref > 0
    t = np.sort(sref)[::-1][keep - 1]
    dist = np.abs(sref - t) / t
    rel = np.zeros_like(sref)
    rel[nz] = np.abs(scores[nz] - sref[nz]) / sref[nz]
    near = nz & (dist < 1e-3)
    say("score rel err: max", f"{rel.max():.2e}", "near the cut", f"{rel[near].max() if near.any() else 0:.2e}")
    assert np.all(rel < np.maximum(dist, TAU) / 4)
    if near.any():
        assert rel[near].max() < TAU / 10


def _case(wl, seed):
    gs = GradientStream(wl, seed=seed)
    return gs.rows(0, wl.m), gs.theta()


@pytest.mark.parametrize("m,B,nb,lam,batch_cap", [
    (100, 256, 6, 1e-3, None),     # m padded to 128 inside
    (64, 512, 3, 1e-4, 2),         # batch boundary inside the block loop
    (1, 64, 4, 1e-2, None),        # m = 1
    (300, 512, 3, 1e-4, None),     # padded to 320: uneven splits in the recursive factor
    (1024, 2048, 3, 1e-4, None),   # the pruning workload's block width and m
    (700, 300, 4, 1e-4, None),     # m > B
    (37, 100, 5, 1e-3, None),      # B not a multiple of the tile widths
    (4096, 1024, 2, 1e-3, None),   # the largest m of the fast mode
    (256, 65536, 1, 1e-4, None),   # the widest block of the fast mode (split Gram)
])
def test_fast_mode_matches_oracle(dev, m, B, nb, lam, batch_cap, monkeypatch):
    """The pruning workload's recipe (entries scaled by 1/sqrt(4,194,304), so
    the Fisher term stays below m*lambda as at full size) at reduced sizes."""
    if batch_cap:
        monkeypatch.setenv("MFAC_STATIC_BATCH_BLOCKS", str(batch_cap))
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=B * nb, m=m, block=B, lam=lam, scale_d=base.d)
    G, theta = _case(wl, seed=41)
    keep = wl.d // 2
    say("fast static", m, B, nb, lam, batch_cap)
    sb, Gd, st, diag, mask, scores = _fast(dev, G, B, lam, theta, keep)
    assert st == 0
    Gn = G.numpy()
    assert np.array_equal(Gd.cpu().numpy(), Gn)          # G left intact
    dref = ostatic.inv_diag(Gn, lam, B)
    assert rel_l2(diag, dref) < 1e-6
    sref = omask.scores(theta.numpy(), dref)
    _certificate(scores, sref, keep)
    np.testing.assert_array_equal(mask, omask.keep_mask(sref, keep))
    # queries form W on first use, from the kept fp32 L^-1
    X = GradientStream(wl, seed=42).queries(0, 2)
    Y = sb.ihvp(X.to(dev)).cpu().numpy()
    Yo = ostatic.ihvp(Gn, lam, B, X.numpy())
    assert max(rel_l2(Y[q], Yo[q]) for q in range(2)) < REL_TOL
    ij = torch.tensor([[0, 0], [0, min(1, wl.d - 1)], [wl.d - 1, wl.d - 1], [B // 2, B // 2 + (B > 1)]])
    el = sb.element(ij).cpu().numpy()
    elo = np.array([ostatic.element(Gn, lam, B, int(i), int(j)) for i, j in ij.tolist()])
    assert np.max(np.abs(el - elo)) < 1e-5 * np.max(np.abs(elo))
    # G is still the input after the queries, so a second mask with other
    # weights is exact as well
    theta2 = GradientStream(wl, seed=43).theta()
    mask2, scores2 = sb.obs_mask(theta2.to(dev), keep // 3)
    torch.cuda.synchronize()
    assert sb.status() == 0
    assert np.array_equal(Gd.cpu().numpy(), Gn)
    s2 = omask.scores(theta2.numpy(), dref)
    np.testing.assert_array_equal(mask2.cpu().numpy(), omask.keep_mask(s2, keep // 3))
    delta = sb.obs_update(theta.to(dev), torch.from_numpy(mask).to(dev)).cpu().numpy()
    dlo = ostatic.obs_update(Gn, lam, B, theta.numpy(), mask)
    assert rel_l2(delta, dlo) < REL_TOL
    assert sb.status() == 0


@pytest.mark.parametrize("keep_frac", [0.0, 1.0, 1.0 / 2048, 0.5, 0.7])
def test_fast_mode_mask_edges_and_ties(dev, keep_frac):
    """keep = 0, d, 1, and cuts inside a band of exactly tied (zero) scores."""
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=8 * 256, m=48, block=256, lam=1e-3, scale_d=base.d)
    G, theta = _case(wl, seed=44)
    theta[::3] = 0.0
    theta[1::7] = -0.0
    keep = int(round(wl.d * keep_frac))
    say("fast mask edges", keep)
    sb, Gd, st, diag, mask, scores = _fast(dev, G, wl.block, wl.lam, theta, keep)
    assert st == 0
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block)
    sref = omask.scores(theta.numpy(), dref)
    np.testing.assert_array_equal(mask, omask.keep_mask(sref, keep))
    assert int(mask.sum()) == keep


def test_fast_mode_dense_near_ties_are_decided_in_fp64(dev):
    """Equal weights everywhere: the mask is decided by the diagonal alone, and
    neighbouring diagonal values are ~1e-7 apart, the size of the fp32 path's
    error. The fp32 scores alone would misorder coordinates at the cut; the
    mask still equals the oracle's, and the scores returned for the band are
    the fp64 values."""
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=32 * 2048, m=256, block=2048, scale_d=base.d)
    G, _ = _case(wl, seed=45)
    theta = torch.full((wl.d,), 0.05, dtype=torch.float32)
    keep = wl.d // 2
    say("fast dense near-ties")
    sb, Gd, st, diag, mask, scores = _fast(dev, G, wl.block, wl.lam, theta, keep)
    assert st == 0
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block)
    sref = omask.scores(theta.numpy(), dref)
    order = np.sort(sref)[::-1]
    gaps = np.diff(order[keep - 50:keep + 50]) / order[keep]
    say("median relative gap near the cut", f"{float(np.median(np.abs(gaps))):.1e}")
    # the band holds more coordinates than the wide refinement's 64 slots, so
    # the single-work-group kernel finishes the rest
    t = order[keep - 1]
    nband = int(np.sum(np.abs(sref - t) <= TAU * t))
    say("band coordinates", nband)
    assert nband > 64
    np.testing.assert_array_equal(mask, omask.keep_mask(sref, keep))
    # the scores closest to the cut are the exact ones
    near = np.argsort(np.abs(sref - order[keep - 1]))[:5]
    assert np.max(np.abs(scores[near] - sref[near]) / sref[near]) < 1e-12


def test_fast_mode_reports_an_uncertified_mask(dev):
    """Blocks whose Fisher term dwarfs m*lambda (per-block entry scale, S_j
    near 1): 1 - S_j cancels and the fp32 diagonal loses digits. The fast mode
    either returns the exact mask or reports MFAC_EPRECISION; never a wrong
    mask with a clean status."""
    from paper_2107_03356_amd import MFAC_EPRECISION
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=8 * 512, m=1500, block=512, lam=1e-5, scale_d=512)
    G, theta = _case(wl, seed=46)
    keep = wl.d // 2
    say("fast mode, ill-conditioned blocks")
    sb, Gd, st, diag, mask, scores = _fast(dev, G, wl.block, wl.lam, theta, keep)
    dref = ostatic.inv_diag(G.numpy(), wl.lam, wl.block)
    exact = np.array_equal(mask, omask.keep_mask(omask.scores(theta.numpy(), dref), keep))
    say("status", st, "mask exact", exact)
    assert st in (0, MFAC_EPRECISION)
    assert exact or st == MFAC_EPRECISION


def test_fast_mode_rejected_where_unsupported(dev):
    from paper_2107_03356_amd import MfacError, StaticBlocks
    G = torch.zeros((4097, 256), device=dev)
    with pytest.raises(MfacError):
        StaticBlocks(G, 256, 1e-3, fp32=True)          # m past the fast mode's limit
    Gh = torch.zeros((8, 1024), pin_memory=True)
    with pytest.raises(MfacError):
        StaticBlocks(Gh, 256, 1e-3, fp32=True, page_cols=512)   # no paged fast mode
