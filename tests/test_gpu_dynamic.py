"""GPU parity of the dynamic sliding-window path against the fp64 oracle.

Every case draws its rows once (synth), hands the same fp32 values to the HIP
path (through the C ABI) and to oracle.dynamic.WindowOracle, and compares
F^-1 g_new (and the fused extra queries) element by element in relative L2.
"""

import numpy as np
import pytest
import torch

from gpu_common import REL_TOL, rel_l2, require_gpu, say
from oracle.dynamic import WindowOracle
from synth import GradientStream, get_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _sliding(dev, wl, seed, nsteps, queries=0, fill_by_replace=False, check=lambda t: True):
    from paper_2107_03356_amd import Window
    gs = GradientStream(wl, seed=seed, device="cpu")
    d, m = wl.d, wl.m
    if fill_by_replace:
        win = Window(d, m, wl.lam, max_queries=queries, device=dev)
        orc = WindowOracle(d, m, wl.lam)
        rows = range(0, m + nsteps)
    else:
        G0 = gs.window()
        win = Window(d, m, wl.lam, max_queries=queries, G0=G0.to(dev), device=dev)
        orc = WindowOracle(d, m, wl.lam, G0=G0.numpy())
        rows = range(m, m + nsteps)
    errs, outs = [], []
    for t, r in enumerate(rows):
        g = gs.row(r)
        if queries:
            X = gs.queries(t, queries)
            y, Y = win.replace(g.to(dev), X=X.to(dev))
        else:
            y = win.replace(g.to(dev))
        slot_before = orc.steps % m
        yo = orc.slide(g.numpy())
        if check(t):
            torch.cuda.synchronize()
            e = rel_l2(y.cpu().numpy(), yo)
            errs.append(e)
            if queries:
                Yo = orc.ihvp(X.numpy())
                for q in range(queries):
                    errs.append(rel_l2(Y[q].cpu().numpy(), Yo[q]))
            assert max(errs[-(1 + queries):]) < REL_TOL, (t, slot_before, errs[-(1 + queries):])
        outs.append(y)
    assert win.status() == 0
    return win, orc, errs, outs


def test_tiny_fill_by_replace_every_step(dev):
    wl = get_workload("dyn_tiny_d4096_m16")
    say("tiny fill_by_replace", wl.d, wl.m)
    win, orc, errs, outs = _sliding(dev, wl, seed=1, nsteps=wl.steps, fill_by_replace=True)
    assert len(errs) == wl.m + wl.steps
    assert max(errs) < 1e-5, max(errs)
    assert win.info() == (0, wl.m + wl.steps)


def test_tiny_init_equals_fill(dev):
    """R2: an empty window filled by m replaces equals init with those rows."""
    wl = get_workload("dyn_tiny_d4096_m16")
    say("tiny init vs fill")
    _, _, errs_a, outs_a = _sliding(dev, wl, seed=2, nsteps=wl.steps, fill_by_replace=True)
    _, _, errs_b, outs_b = _sliding(dev, wl, seed=2, nsteps=wl.steps, fill_by_replace=False)
    assert max(errs_b) < 1e-5
    for ya, yb in zip(outs_a[wl.m:], outs_b):
        assert rel_l2(ya.cpu().numpy(), yb.cpu().numpy()) < 1e-5


@pytest.mark.parametrize("d,m,lam,q,dist", [
    (3 * 2048 + 777, 40, 1e-3, 3, "gauss"),        # ragged d (d % 4 != 0), m not a multiple of 64
    (20000, 200, 1e-4, 2, "lognormal"),            # several 64-wide leaves in the recursive factor
    (30000, 300, 1e-4, 2, "lognormal"),            # padded to 320: uneven splits and half tiles in the factor
    (24000, 1500, 1e-4, 3, "lognormal"),           # m > 1024: padded to 1536, 12 Gram tiles, deeper recursion
    (40968, 1024, 1e-5, 8, "lognormal"),           # m = 1024 with 8 fused queries (ResNet18 recipe)
    (2048, 1, 1e-2, 1, "gauss"),                   # m = 1 (Sherman-Morrison)
    (5, 3, 1e-1, 1, "gauss"),                      # d smaller than one float4 group row
    (8192, 4096, 1e-3, 1, "gauss"),                # m = 4096: 528 Gram tiles, six recursion levels
    (12000, 1500, 1e-4, 9, "lognormal"),           # 10 vectors at m = 1500: pass-2 coefficient rows left unpadded (LDS bound)
    (9000, 300, 1e-4, 16, "gauss"),                # the most fused vectors (17), padded rows of 20
    (4000, 5461, 1e-2, 2, "gauss"),                # 3 vectors at the largest m (m * 3 = 16383): fp64 LDS rows
])
def test_ragged_and_multitile_with_queries(dev, d, m, lam, q, dist):
    base = get_workload("dyn_resnet18_d11.2m_m1024_q8")
    wl = base.scaled(d=d, m=m, lam=lam, dist=dist, queries=q, scale_d=(base.d if dist == "lognormal" else 0))
    say("ragged", d, m, lam, q)
    nsteps = 6 if m >= 1024 else 12
    _, _, errs, _ = _sliding(dev, wl, seed=3, nsteps=nsteps, queries=q)
    assert max(errs) < REL_TOL


def test_d1m_m256_full_size(dev):
    """The d = 1,048,576, m = 256 workload at full size (a few sliding steps)."""
    wl = get_workload("dyn_d1m_m256")
    say("d1m m256 full size")
    _, _, errs, _ = _sliding(dev, wl, seed=0, nsteps=4)
    assert max(errs) < REL_TOL


def test_largest_window_m16384(dev):
    """The largest window the library accepts without queries (m = 16384: the
    fp64 pass-1 row sums fill 128 KB of LDS), over a short d; two sliding steps."""
    base = get_workload("dyn_tiny_d4096_m16")
    wl = base.scaled(d=2048, m=16384, lam=1e-2, fill_by_replace=False)
    say("largest window m16384")
    _, _, errs, _ = _sliding(dev, wl, seed=5, nsteps=2)
    assert max(errs) < REL_TOL


def test_correlated_rows_resnet50_recipe_small(dev):
    """10% correlated rows (ResNet50 recipe) at reduced d, full m = 1024."""
    base = get_workload("dyn_resnet50_d25.6m_m1024")
    wl = base.scaled(d=65536, scale_d=base.d)
    say("resnet50 recipe small")
    _, _, errs, _ = _sliding(dev, wl, seed=0, nsteps=4)
    assert max(errs) < REL_TOL


def test_ihvp_and_explicit_slots(dev):
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=30000, m=96, scale_d=base.d)
    gs = GradientStream(wl, seed=5)
    G0 = gs.window()
    say("ihvp + explicit slots")
    win = Window(wl.d, wl.m, wl.lam, max_queries=4, G0=G0.to(dev), device=dev)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    X = gs.queries(0, 4)
    Y = win.ihvp(X.to(dev))
    Yo = orc.ihvp(X.numpy())
    for q in range(4):
        assert rel_l2(Y[q].cpu().numpy(), Yo[q]) < REL_TOL
    # explicit slots, in a non-ring order; ring head must not move
    for t, slot in enumerate([17, 3, 95, 3, 0]):
        g = gs.row(wl.m + t)
        y = win.replace(g.to(dev), slot=slot)
        orc.replace(slot, g.numpy())
        assert rel_l2(y.cpu().numpy(), orc.ihvp(g.numpy())) < REL_TOL
    assert win.info() == (0, 5)
    np.testing.assert_array_equal(win.get_rows().cpu().numpy(), orc.G)
    Y = win.ihvp(X[:1].to(dev).contiguous())
    assert rel_l2(Y[0].cpu().numpy(), orc.ihvp(X[0].numpy())) < REL_TOL


def test_replace_without_output_and_queries_only(dev):
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=12345 * 4, m=70, scale_d=base.d)
    gs = GradientStream(wl, seed=6)
    G0 = gs.window()
    say("replace without y_out")
    win = Window(wl.d, wl.m, wl.lam, max_queries=2, G0=G0.to(dev), device=dev)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    g = gs.row(wl.m)
    win.replace(g.to(dev), want_y=False)          # window update only
    orc.slide(g.numpy())
    g2 = gs.row(wl.m + 1)
    X = gs.queries(1, 2)
    _, Y = win.replace(g2.to(dev), X=X.to(dev), want_y=False)   # queries but no y_out
    orc.slide(g2.numpy())
    Yo = orc.ihvp(X.numpy())
    for q in range(2):
        assert rel_l2(Y[q].cpu().numpy(), Yo[q]) < REL_TOL


def test_deterministic_bitwise(dev):
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=50000, m=128, scale_d=base.d)
    say("determinism")
    _, _, _, a = _sliding(dev, wl, seed=7, nsteps=5, queries=0, check=lambda t: False)
    _, _, _, b = _sliding(dev, wl, seed=7, nsteps=5, queries=0, check=lambda t: False)
    for ya, yb in zip(a, b):
        assert torch.equal(ya, yb)


def test_checkpoint_resume(dev):
    """Resume = init from the saved rows + head; continues like the original."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=40000, m=64, scale_d=base.d)
    gs = GradientStream(wl, seed=8)
    G0 = gs.window()
    say("checkpoint/resume")
    win = Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev)
    for t in range(5):
        win.replace(gs.row(wl.m + t).to(dev))
    rows = win.get_rows()
    head, steps = win.info()
    win2 = Window(wl.d, wl.m, wl.lam, G0=rows, device=dev)
    win2.set_head(head, steps)
    for t in range(5, 9):
        g = gs.row(wl.m + t).to(dev)
        ya, yb = win.replace(g), win2.replace(g)
        assert rel_l2(ya.cpu().numpy(), yb.cpu().numpy()) < 1e-5
    assert win.info() == win2.info()


def test_checkpoint_resume_bitwise_after_rebuild(dev):
    """The derived state (K, the explicit inverse, the refactor counter) is
    rebuilt from the rows on resume; rebuilding the original at the
    checkpoint too makes both continue bitwise identically."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=40000, m=64, scale_d=base.d)
    gs = GradientStream(wl, seed=10)
    say("checkpoint/resume bitwise")
    win = Window(wl.d, wl.m, wl.lam, G0=gs.window().to(dev), device=dev)
    for t in range(5):
        win.replace(gs.row(wl.m + t).to(dev))
    rows = win.get_rows()
    head, steps = win.info()
    win.rebuild()
    win2 = Window(wl.d, wl.m, wl.lam, G0=rows, device=dev)
    win2.set_head(head, steps)
    for t in range(5, 12):
        g = gs.row(wl.m + t).to(dev)
        assert torch.equal(win.replace(g), win2.replace(g))
    assert win.info() == win2.info()
    assert win.status() == 0 and win2.status() == 0


def test_nonfinite_latched_and_rebuild_recovers(dev):
    from paper_2107_03356_amd import MFAC_ENONFINITE, Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=8192, m=32, scale_d=base.d)
    gs = GradientStream(wl, seed=9)
    G0 = gs.window()
    say("non-finite latch")
    win = Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev)   # max_queries = 0: ihvp still takes 1 vector
    bad = gs.row(wl.m).clone()
    bad[100] = float("nan")
    win.replace(bad.to(dev), slot=4)
    assert win.status() == MFAC_ENONFINITE
    assert win.status() == 0          # cleared after being reported
    good = gs.row(wl.m + 1)
    win.set_rows(4, good[None, :].to(dev).contiguous())
    win.rebuild()
    assert win.status() == 0
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    orc.replace(4, good.numpy())
    x = gs.queries(0, 1)
    y = win.ihvp(x.to(dev))
    assert rel_l2(y[0].cpu().numpy(), orc.ihvp(x[0].numpy())) < REL_TOL


@pytest.mark.parametrize("period", [0, 1, 3])
def test_refactor_policies(dev, period):
    """Per-replace refactor (period 0/1) and a refactor every 3 replaces agree with the oracle."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=9000, m=80, scale_d=base.d)
    gs = GradientStream(wl, seed=13)
    G0 = gs.window()
    say("refactor policy", period)
    win = Window(wl.d, wl.m, wl.lam, max_queries=2, G0=G0.to(dev), device=dev)
    win.set_refactor_period(period)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    for t in range(10):
        g = gs.row(wl.m + t)
        X = gs.queries(t, 2)
        y, Y = win.replace(g.to(dev), X=X.to(dev))
        yo = orc.slide(g.numpy())
        Yo = orc.ihvp(X.numpy())
        assert rel_l2(y.cpu().numpy(), yo) < REL_TOL
        assert max(rel_l2(Y[q].cpu().numpy(), Yo[q]) for q in range(2)) < REL_TOL
    assert win.status() == 0


@pytest.mark.parametrize("m", [150, 300, 448, 520, 700, 1030])
def test_refactor_every_replace_across_gemm_tile_paths(dev, m):
    """A refactor on every replace at window sizes whose factor takes each
    GEMM path of one matrix: 64 x 64 tiles only (m = 150, 300: padded to
    192, 320), a product exactly 256 wide (448), 128 x 128 tiles with half
    tiles beside 64 x 64 ones (520 -> 576, 700 -> 704), and m > 1024
    (1030 -> 1088); one matrix always splits K over several work-groups."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wl = base.scaled(d=12000 + 37, m=m, scale_d=base.d)
    gs = GradientStream(wl, seed=21)
    G0 = gs.window()
    say("refactor every replace, m", m)
    win = Window(wl.d, wl.m, wl.lam, max_queries=1, G0=G0.to(dev), device=dev)
    win.set_refactor_period(0)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    worst = 0.0
    for t in range(3):
        g = gs.row(wl.m + t)
        X = gs.queries(t, 1)
        y, Y = win.replace(g.to(dev), X=X.to(dev))
        yo = orc.slide(g.numpy())
        Yo = orc.ihvp(X.numpy())
        worst = max(worst, rel_l2(y.cpu().numpy(), yo), rel_l2(Y[0].cpu().numpy(), Yo[0]))
    say("worst rel L2", f"{worst:.2e}")
    assert win.status() == 0
    # well conditioned (m < d, lambda = 1e-4) with fp64 coefficients: what is
    # left is the fp32 rounding of the data (~3e-8), so a factor that is off
    # in any tile shows far below the general 1e-4 bar
    assert worst < 1e-6


def test_long_run_inverse_updates_do_not_drift(dev):
    """400 O(m^2) inverse updates (over six trips round a 64-slot ring) without a refactor."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_resnet50_d25.6m_m1024")
    wl = base.scaled(d=16384, m=64, lam=1e-4, scale_d=base.d // 64)
    gs = GradientStream(wl, seed=14)
    G0 = gs.window()
    say("long run drift")
    win = Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev)
    win.set_refactor_period(100000)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    errs = []
    for t in range(400):
        g = gs.row(wl.m + t)
        y = win.replace(g.to(dev))
        yo = orc.slide(g.numpy())
        if t % 25 == 24:
            errs.append(rel_l2(y.cpu().numpy(), yo))
    assert win.status() == 0
    assert max(errs) < 1e-5, errs


@pytest.mark.parametrize("d,m,lam,q", [
    (96, 256, 1e-6, 0),      # m > d: K has rank 96 of 256, A's condition number ~1e5
    (300, 512, 1e-7, 0),     # rank 300 of 512, condition number ~1e6
    (96, 256, 1e-6, 3),      # the same with 3 fused queries (4 vectors: fp64 passes)
])
def test_rank_deficient_window_long_run(dev, d, m, lam, q):
    """More gradients than coordinates and a small damping: A = K + m*lambda*I
    is ill-conditioned; 700 replaces of O(m^2) inverse updates, no refactor.
    With fp32 sums in the passes the IHVP error grows with the condition
    number (1e-3 here); fp64 sums keep it at the fp32 rounding of the data."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_tiny_d4096_m16")
    wl = base.scaled(d=d, m=m, lam=lam, fill_by_replace=False)
    gs = GradientStream(wl, seed=15)
    G0 = gs.window()
    say("rank-deficient long run", d, m, lam, q)
    win = Window(wl.d, wl.m, wl.lam, max_queries=q, G0=G0.to(dev), device=dev)
    win.set_refactor_period(100000)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    errs = []
    for t in range(700):
        g = gs.row(wl.m + t)
        check = t % 50 == 49
        if q:
            X = gs.queries(t, q)
            y, Y = win.replace(g.to(dev), X=X.to(dev))
        else:
            y = win.replace(g.to(dev))
        yo = orc.slide(g.numpy())
        if check:
            errs.append(rel_l2(y.cpu().numpy(), yo))
            if q:
                Yo = orc.ihvp(X.numpy())
                errs += [rel_l2(Y[j].cpu().numpy(), Yo[j]) for j in range(q)]
    assert win.status() == 0
    assert max(errs) < 1e-5, max(errs)


@pytest.mark.parametrize("d,m", [
    (3 * 2048 + 5, 1),       # one row: three of the four waves fold nothing
    (1000, 3),               # d below one slab, m < 4
    (4 * 2048 + 777, 7),     # ragged last slab (d % 4 != 0)
    (6000, 4096),            # the largest m of the one-vector split-row pass 2 (160 KB of LDS)
])
def test_single_vector_pass2_shapes(dev, d, m):
    """One inserted gradient and no queries (the one-vector pass 2), with
    its output at an unaligned address (scalar tail stores) on one step, and
    a one-vector IHVP (reads x, alpha = 1/lambda) with an unaligned output."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_tiny_d4096_m16")
    wl = base.scaled(d=d, m=m, lam=1e-2, fill_by_replace=False)
    gs = GradientStream(wl, seed=17)
    G0 = gs.window()
    say("single-vector pass 2", d, m)
    win = Window(wl.d, wl.m, wl.lam, max_queries=0, G0=G0.to(dev), device=dev)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    buf = torch.full((d + 1,), float("nan"), device=dev)
    for t in range(3):
        g = gs.row(m + t)
        y = win.replace(g.to(dev), y_out=buf[1:] if t == 1 else None)
        yo = orc.slide(g.numpy())
        assert rel_l2(y.cpu().numpy(), yo) < REL_TOL, t
    assert torch.isnan(buf[0]).item()                       # nothing written before the output
    x = gs.queries(0, 1)[0]
    xo = orc.ihvp(x[None].numpy())[0]
    assert rel_l2(win.ihvp(x.to(dev)).cpu().numpy(), xo) < REL_TOL
    buf2 = torch.full((d + 1,), float("nan"), device=dev)
    y2 = win.ihvp(x.to(dev), Y=buf2[1:])
    assert rel_l2(y2.cpu().numpy(), xo) < REL_TOL
    assert torch.isnan(buf2[0]).item()
    assert win.status() == 0


def test_default_policy_over_a_refactor_boundary_m1024(dev):
    """m = 1024 with the default coefficient policy (O(m^2) inverse updates,
    full refactor every 1024 replaces): 1100 steps, checked right before,
    at and after the refactor and at the end."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_resnet50_d25.6m_m1024")
    wl = base.scaled(d=8192, scale_d=base.d)
    gs = GradientStream(wl, seed=21, device="cpu")
    G0 = gs.window()
    win = Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    checked = {0, 1, 511, 1021, 1022, 1023, 1024, 1025, 1099}
    say("default policy over a refactor boundary, m = 1024")
    errs = []
    for t in range(1100):
        g = gs.row(wl.m + t)
        y = win.replace(g.to(dev))
        if t in checked:
            yo = orc.slide(g.numpy())
            errs.append(rel_l2(y.cpu().numpy(), yo))
            assert errs[-1] < REL_TOL, (t, errs[-1])
        else:
            orc.replace(orc.steps % wl.m, g.numpy())
    assert win.status() == 0
    assert win.info() == (1100 % wl.m, 1100)


def test_default_policy_m1024_at_resnet50_conditioning(dev):
    """The ResNet50 window's conditioning at a size the oracle can follow for
    1100 steps: m = 1024, lambda = 1e-5, log-normal scales with 10% correlated
    rows, and entries scaled by 1/sqrt(d) of this d, so |g|^2 / (m lambda) is
    about 720 as in the full-size workload (the Fisher term far above the
    damping). Default coefficient policy: O(m^2) inverse updates with the
    scheduled refactor after 1024 replaces; checked early, every 100 steps,
    right before, at and after the refactor, and at the end."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_resnet50_d25.6m_m1024")
    d = 12000
    wl = base.scaled(d=d, scale_d=d)
    assert wl.corr_frac == 0.1 and wl.lam == 1e-5 and wl.m == 1024
    gs = GradientStream(wl, seed=24, device="cpu")
    G0 = gs.window()
    ratio = float((G0.double() ** 2).sum(1).mean()) / (wl.m * wl.lam)
    assert 300 < ratio < 3000, ratio
    win = Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev)
    orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
    checked = {0, 1, 2, 1021, 1022, 1023, 1024, 1025, 1099} | set(range(99, 1100, 100))
    say("default policy at the ResNet50 conditioning, m = 1024, d =", d, "|g|^2/(m lambda) =", round(ratio))
    errs = {}
    for t in range(1100):
        g = gs.row(wl.m + t)
        y = win.replace(g.to(dev))
        if t in checked:
            yo = orc.slide(g.numpy())
            errs[t] = rel_l2(y.cpu().numpy(), yo)
            assert errs[t] < REL_TOL, (t, errs[t])
        else:
            orc.replace(orc.steps % wl.m, g.numpy())
    assert win.status() == 0
    say("errors", {k: f"{v:.1e}" for k, v in sorted(errs.items())})
    # no growth over the 1023 updates before the refactor beyond fp32 rounding
    assert max(errs.values()) < 1e-5, errs


def test_two_windows_on_two_streams_interleaved(dev):
    """Handles are independent: two windows, each bound to its own stream,
    replaced alternately without host synchronisation, both match their oracles."""
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_d1m_m256")
    wls = [base.scaled(d=20000, m=48, scale_d=base.d), base.scaled(d=13001, m=70, scale_d=base.d)]
    streams = [torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)]
    say("two windows on two streams")
    wins, orcs, gss, outs = [], [], [], [[], []]
    for i, wl in enumerate(wls):
        gs = GradientStream(wl, seed=50 + i)
        G0 = gs.window()
        with torch.cuda.stream(streams[i]):
            wins.append(Window(wl.d, wl.m, wl.lam, G0=G0.to(dev), device=dev))
        orcs.append(WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy()))
        gss.append(gs)
    torch.cuda.synchronize()
    for t in range(6):
        for i in range(2):
            g = gss[i].row(wls[i].m + t)
            with torch.cuda.stream(streams[i]):
                outs[i].append((wins[i].replace(g.to(dev, non_blocking=False)), g))
    torch.cuda.synchronize()
    for i in range(2):
        for y, g in outs[i]:
            yo = orcs[i].slide(g.numpy())
            assert rel_l2(y.cpu().numpy(), yo) < REL_TOL
        assert wins[i].status() == 0


def test_step_cost_is_linear_in_d_and_coefficients_independent_of_d(dev):
    """The complexity claims of Section 3.2: the two passes cost O(dm) (4x the
    columns, ~4x the pass time) and the coefficient phase O(m^2), independent
    of d. Phase times from the library's own HIP-event tracing."""
    from paper_2107_03356_amd import Window
    m = 256
    phases = {}
    for d in (1 << 21, 1 << 23):
        say("complexity", d, m)
        win = Window(d, m, 1e-4, device=dev)
        gen = torch.Generator(device=dev)
        gen.manual_seed(d)
        g = torch.randn((24, d), device=dev, generator=gen) / d ** 0.5
        for t in range(4):
            win.replace(g[t])
        torch.cuda.synchronize()
        win.trace_read()
        win.trace(True)
        for t in range(4, 24):
            win.replace(g[t])
        torch.cuda.synchronize()
        win.trace(False)
        ms, cnt = win.trace_read()
        phases[d] = [ms[i] / max(cnt[i], 1) for i in range(4)]
        assert win.status() == 0
        win.close()
    small, big = phases[1 << 21], phases[1 << 23]
    passes = (big[0] + big[2]) / (small[0] + small[2])
    coef = big[1] / small[1]
    assert 3.0 < passes < 5.5, (passes, small, big)
    assert 0.5 < coef < 2.0, (coef, small, big)
