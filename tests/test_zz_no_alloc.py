"""mfac_ihvp_noalloc (the allocation-free IHVP) against mfac_ihvp, through the C ABI.

Two calls in a row on one window (four vectors, then one: the second call
reads less than the first left in the shared scratch), then a call on a
second, smaller window, each compared with the existing entry point on the
same inputs and with the fp64 oracle; and the size limit rejected on the
host before anything is enqueued.
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


def _both(B, win, X):
    """(Y from mfac_ihvp, Y from mfac_ihvp_noalloc) for the rows of X."""
    n = X.shape[0]
    Y1 = torch.full_like(X, float("nan"))
    Y2 = torch.full_like(X, float("nan"))
    assert B.mfac_ihvp(win.handle, n, X.data_ptr(), Y1.data_ptr()) == B.MFAC_OK
    assert B.mfac_ihvp_noalloc(win.handle, n, X.data_ptr(), Y2.data_ptr()) == B.MFAC_OK
    torch.cuda.synchronize()
    assert win.status() == 0
    return Y1.cpu().numpy(), Y2.cpu().numpy()


def test_noalloc_ihvp_matches_ihvp_and_oracle(dev):
    from paper_2107_03356_amd import Window
    from paper_2107_03356_amd import _binding as B
    base = get_workload("dyn_d1m_m256")
    cases = [(base.scaled(d=70001, m=300, scale_d=base.d), 4, 31),   # first call: 4 vectors
             (None, 1, None),                                         # same window, 1 vector
             (base.scaled(d=9000, m=37, scale_d=base.d), 2, 32)]      # a smaller window
    win = orc = gs = None
    for wl, n, seed in cases:
        if wl is not None:
            gs = GradientStream(wl, seed=seed)
            G0 = gs.window()
            say("noalloc ihvp: window d =", wl.d, "m =", wl.m)
            win = Window(wl.d, wl.m, wl.lam, max_queries=3, G0=G0.to(dev), device=dev)
            orc = WindowOracle(wl.d, wl.m, wl.lam, G0=G0.numpy())
        say("noalloc ihvp: n =", n)
        X = gs.queries(n, n)
        Y1, Y2 = _both(B, win, X.to(dev).contiguous())
        Yo = orc.ihvp(X.numpy())
        for q in range(n):
            assert rel_l2(Y2[q], Y1[q]) < REL_TOL, (n, q)
            assert rel_l2(Y2[q], Yo[q]) < REL_TOL, (n, q)
        # the same kernels in the same order: the two entry points agree bitwise
        assert np.array_equal(Y1, Y2)


def test_noalloc_ihvp_rejects_sizes_past_its_scratch(dev):
    """m * n beyond the 16 MiB scratch: MFAC_EWORKSPACE, nothing written."""
    from paper_2107_03356_amd import Window
    from paper_2107_03356_amd import _binding as B
    d, m = 3000, 4081
    say("noalloc ihvp: limit, m =", m)
    win = Window(d, m, 1e-2, max_queries=0, device=dev)
    X = torch.ones((1, d), device=dev)
    Y = torch.full_like(X, float("nan"))
    assert B.mfac_ihvp_noalloc(win.handle, 1, X.data_ptr(), Y.data_ptr()) == B.MFAC_EWORKSPACE
    torch.cuda.synchronize()
    assert torch.isnan(Y).all().item()
    # one row less fits (m * n = 4080)
    win2 = Window(d, m - 1, 1e-2, max_queries=0, device=dev)
    assert B.mfac_ihvp_noalloc(win2.handle, 1, X.data_ptr(), Y.data_ptr()) == B.MFAC_OK
    torch.cuda.synchronize()
    assert win2.status() == 0
    # an empty window is lambda^-1 I
    np.testing.assert_allclose(Y.cpu().numpy(), 100.0, rtol=1e-6)
    win.close()
    win2.close()
