"""GPU parity of mfac_window_replace_seq (a sequence of sliding steps whose
gradients are known in advance: each step's IHVP pass also forms the next
gradient's Gram column) against the fp64 oracle and against the same steps
made one mfac_window_replace at a time."""

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


def _case(dev, d, m, lam, n, dist, from_empty, seed=5, chunks=(None,), period=None):
    from paper_2107_03356_amd import Window
    base = get_workload("dyn_resnet18_d11.2m_m1024_q8")
    wl = base.scaled(d=d, m=m, lam=lam, dist=dist, queries=0, scale_d=(base.d if dist == "lognormal" else 0))
    gs = GradientStream(wl, seed=seed, device="cpu")
    if from_empty:
        G0, r0 = None, 0
    else:
        G0, r0 = gs.window(), m
    Gn = gs.rows(r0, n).contiguous()
    seq = Window(d, m, lam, G0=None if G0 is None else G0.to(dev), device=dev)
    one = Window(d, m, lam, G0=None if G0 is None else G0.to(dev), device=dev)
    orc = WindowOracle(d, m, lam, G0=None if G0 is None else G0.numpy())
    if period is not None:
        seq.set_refactor_period(period)
        one.set_refactor_period(period)
    Gd = Gn.to(dev)
    # the sequence in one call, or in consecutive calls of the given lengths
    Ys, t0 = [], 0
    for c in chunks:
        c = n - t0 if c is None else c
        Ys.append(seq.replace_seq(Gd[t0:t0 + c]))
        t0 += c
    Y = torch.cat(Ys)
    torch.cuda.synchronize()
    worst_orc, worst_one = 0.0, 0.0
    for t in range(n):
        yo = orc.slide(Gn[t].numpy())
        y1 = one.replace(Gd[t])
        worst_orc = max(worst_orc, rel_l2(Y[t].cpu().numpy(), yo))
        worst_one = max(worst_one, rel_l2(Y[t].cpu().numpy(), y1.cpu().numpy()))
    assert seq.status() == 0 and one.status() == 0
    assert seq.info() == one.info()
    # the window state after the sequence serves later single replaces
    g = gs.row(r0 + n)
    y_after = seq.replace(g.to(dev))
    yo = orc.slide(g.numpy())
    return worst_orc, worst_one, rel_l2(y_after.cpu().numpy(), yo)


@pytest.mark.parametrize("d,m,lam,n,dist,from_empty", [
    (4096, 16, 1e-3, 40, "gauss", True),          # fill from zeros, then wrap the ring
    (5003, 37, 1e-3, 50, "gauss", False),         # ragged d (no 16-byte rows), m not a multiple of 4 or 32
    (3000, 1, 1e-2, 6, "gauss", False),           # m = 1: the next gradient replaces the row just read
    (4100, 3, 1e-2, 9, "gauss", False),           # fewer rows than waves
    (2048 * 300 + 7, 64, 1e-4, 6, "lognormal", False),  # more slabs than work-groups
    (6244, 2048, 1e-3, 3, "gauss", False),        # the largest fused m (160 KB of LDS)
    (4096, 2049, 1e-3, 3, "gauss", False),        # above it: two passes per step
    (40968, 1024, 1e-5, 5, "lognormal", False),   # the headline m, ragged d
])
def test_replace_seq_matches_oracle_and_single_replaces(dev, d, m, lam, n, dist, from_empty):
    say("replace_seq", d, m, lam, n, from_empty)
    e_orc, e_one, e_after = _case(dev, d, m, lam, n, dist, from_empty)
    assert e_orc < REL_TOL, e_orc
    # same coefficients up to the order of the fp64 sums in the Gram column
    assert e_one < 1e-6, e_one
    assert e_after < REL_TOL, e_after


def test_replace_seq_in_chunks_and_length_one(dev):
    say("replace_seq chunks", 4096, 16)
    e_orc, e_one, e_after = _case(dev, 4096, 16, 1e-3, 23, "gauss", False, chunks=(1, 7, 1, None))
    assert e_orc < REL_TOL and e_one < 1e-6 and e_after < REL_TOL, (e_orc, e_one, e_after)


def test_replace_seq_rejects_bad_arguments(dev):
    from paper_2107_03356_amd import _binding as B
    from paper_2107_03356_amd import Window
    say("replace_seq arguments")
    w = Window(4096, 8, 1e-3, device=dev)
    G = torch.zeros(2, 4096, device=dev)
    lib = B.load()
    assert lib.mfac_window_replace_seq(w.handle, 0, G.data_ptr(), G.data_ptr()) == B.MFAC_EINVAL
    assert lib.mfac_window_replace_seq(w.handle, 2, None, G.data_ptr()) == B.MFAC_EINVAL
    assert lib.mfac_window_replace_seq(w.handle, 2, G.data_ptr() + 2, G.data_ptr()) == B.MFAC_EINVAL
    assert w.info() == (0, 0)
    assert w.status() == 0


@pytest.mark.parametrize("period", [0, 2, 5])
def test_replace_seq_under_refactor_policies(dev, period):
    """Refactor on every replace, every second, every fifth: the sequence
    takes the same coefficient path per step as single replaces."""
    say("replace_seq refactor period", period)
    e_orc, e_one, e_after = _case(dev, 6000, 24, 1e-3, 17, "gauss", False, period=period)
    assert e_orc < REL_TOL and e_one < 1e-6 and e_after < REL_TOL, (e_orc, e_one, e_after)


@pytest.mark.parametrize("m,fused", [(16, True), (2049, False)])
def test_replace_seq_phase_trace_counts(dev, m, fused):
    from paper_2107_03356_amd import Window
    say("replace_seq trace", m)
    d, n = 4096, 5
    w = Window(d, m, 1e-3, device=dev)
    Gn = torch.randn(n, d, device=dev) / 64.0
    w.trace(True)
    w.replace_seq(Gn)
    w.trace(False)
    ms, cnt = w.trace_read()
    # phases: 0 pass 1, 1 coefficients, 2 pass 2 (fused with the next pass 1), 3 row write
    assert cnt == [1 if fused else n, n, n, n], cnt
    assert all(t >= 0.0 for t in ms)
    assert w.status() == 0
    assert w.info() == (n % m, n)
