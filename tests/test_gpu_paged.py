"""GPU parity of the host-paged static precompute (Appendix C's host paging).

G lives in pinned host memory and passes through the device in column pages.
Block-wise pages hold whole blocks and run the same kernels on the same data
as the on-device path, so their W and diagonal must be bitwise equal to it;
a single block spanning d sums its Gram page by page (a different rounding
order), so it is compared with the fp64 oracle.
"""

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
    m, d = G.shape
    out = np.empty((m, d))
    for b in range(d // B):
        Gb = G[:, b * B:(b + 1) * B].astype(np.float64)
        R = np.linalg.cholesky(Gb @ Gb.T + m * lam * np.eye(m))
        out[:, b * B:(b + 1) * B] = sla.solve_triangular(R, Gb, lower=True)
    return out


def _problem(m, B, d, lam, seed):
    base = get_workload("static_d4.19m_b2048_m1024")
    wl = base.scaled(d=d, m=m, block=B, lam=lam, scale_d=B)
    gs = GradientStream(wl, seed=seed)
    return wl, gs.rows(0, m), gs.theta()


def _pinned(G):
    P = torch.empty(G.shape, dtype=torch.float32, pin_memory=True)
    P.copy_(G)
    return P


@pytest.mark.parametrize("m,B,nb,page_blocks", [
    (100, 256, 7, 2),      # 4 pages, the last with one block
    (64, 512, 5, 5),       # one page holding every block
    (300, 512, 3, 1),      # one block per page, m padded to 320
])
def test_blockwise_pages_equal_the_device_path(dev, m, B, nb, page_blocks):
    from paper_2107_03356_amd import StaticBlocks
    wl, G, theta = _problem(m, B, B * nb, 1e-4, seed=51)
    say("paged block-wise", m, B, nb, page_blocks)
    Gh = _pinned(G)
    sp = StaticBlocks(Gh, B, wl.lam, page_cols=B * page_blocks, device=dev)
    d64p = sp.inv_diag(fp64=True)
    maskp, scp = sp.obs_mask(theta.to(dev), wl.d // 2)
    torch.cuda.synchronize()
    assert sp.status() == 0
    Gd = G.to(dev).contiguous()
    sd = StaticBlocks(Gd, B, wl.lam)
    d64 = sd.inv_diag(fp64=True)
    torch.cuda.synchronize()
    assert sd.status() == 0
    assert torch.equal(d64p, d64)
    assert torch.equal(Gh, Gd.cpu())                      # W written back over the host G
    dref = ostatic.inv_diag(G.numpy(), wl.lam, B)
    assert rel_l2(d64p.cpu().numpy(), dref) < 1e-11
    assert rel_l2(Gh.numpy(), _oracle_W(G.numpy(), wl.lam, B)) < 1e-6
    sref = omask.scores(theta.numpy(), dref)
    np.testing.assert_array_equal(maskp.cpu().numpy(), omask.keep_mask(sref, wl.d // 2))


@pytest.mark.parametrize("m,d,page_cols", [
    (64, 20000, 4096),     # 5 pages: split Gram summed over pages, a ragged last page
    (130, 9000, 9000),     # one page (m padded to 192)
    (256, 65536, 8192),    # 8 pages of 8192 columns, 4 column splits each
])
def test_full_d_pages_match_the_oracle(dev, m, d, page_cols):
    from paper_2107_03356_amd import StaticBlocks
    wl, G, theta = _problem(m, d, d, 1e-4, seed=52)
    say("paged full-d", m, d, page_cols)
    Gh = _pinned(G)
    sp = StaticBlocks(Gh, d, wl.lam, page_cols=page_cols, device=dev, trace=True)
    d64 = sp.inv_diag(fp64=True)
    mask, sc = sp.obs_mask(theta.to(dev), d // 2)
    torch.cuda.synchronize()
    assert sp.status() == 0
    ms, cnt = sp.trace_read()
    npages = -(-d // page_cols)
    assert cnt[:3] == [npages, 1, npages]
    dref = ostatic.inv_diag(G.numpy(), wl.lam, d)
    assert rel_l2(d64.cpu().numpy(), dref) < 1e-11
    assert rel_l2(Gh.numpy(), _oracle_W(G.numpy(), wl.lam, d)) < 1e-6
    sref = omask.scores(theta.numpy(), dref)
    assert rel_l2(sc.cpu().numpy(), sref) < 1e-11
    np.testing.assert_array_equal(mask.cpu().numpy(), omask.keep_mask(sref, d // 2))


def test_queries_read_w_from_host_memory(dev):
    """IHVP, element and OBS queries of a paged handle against the oracle."""
    from paper_2107_03356_amd import StaticBlocks
    wl, G, theta = _problem(96, 512, 4 * 512, 1e-3, seed=53)
    X = GradientStream(wl, seed=53).queries(0, 3)
    say("paged queries")
    Gh = _pinned(G)
    sp = StaticBlocks(Gh, wl.block, wl.lam, page_cols=1024, device=dev)
    Y = sp.ihvp(X.to(dev).contiguous())
    Yo = ostatic.ihvp(G.numpy(), wl.lam, wl.block, X.numpy())
    for q in range(3):
        assert rel_l2(Y[q].cpu().numpy(), Yo[q]) < 1e-4
    pairs = [(0, 0), (5, 17), (511, 3), (600, 1000), (2047, 2040), (3, 900)]
    el = sp.element(torch.tensor(pairs, dtype=torch.int64)).cpu().numpy()
    ref = np.array([ostatic.element(G.numpy(), wl.lam, wl.block, i, j) for i, j in pairs])
    assert np.max(np.abs(el - ref)) < 1e-5 * np.abs(ref).max()
    mask, _ = sp.obs_mask(theta.to(dev), wl.d // 2)
    delta = sp.obs_update(theta.to(dev), mask)
    torch.cuda.synchronize()
    assert sp.status() == 0
    dref = ostatic.obs_update(G.numpy(), wl.lam, wl.block, theta.numpy(), mask.cpu().numpy())
    assert rel_l2(delta.cpu().numpy(), dref) < 1e-4


def test_pageable_host_memory_is_rejected(dev):
    """The binding refuses an unpinned tensor, and the C entry point refuses
    pageable memory by itself."""
    import ctypes

    from paper_2107_03356_amd import MFAC_EINVAL, StaticBlocks, load
    G = torch.zeros((8, 1024), dtype=torch.float32)
    with pytest.raises(ValueError):
        StaticBlocks(G, 256, 1e-3, page_cols=512, device=dev)
    lib = load()
    wb = lib.mfac_static_paged_workspace_bytes(1024, 256, 8, 512)
    ws = torch.empty(wb, dtype=torch.uint8, device=dev)
    h = ctypes.c_void_p()
    st = lib.mfac_static_precompute_paged(ctypes.byref(h), 1024, 256, 8, 1e-3, G.data_ptr(), 512, ws.data_ptr(),
                                          wb, 0, None)
    assert st == MFAC_EINVAL and h.value is None
