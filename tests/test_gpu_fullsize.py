"""Full-size parity, in the launch configuration bench.py times.

Dynamic: the ResNet50-sized window (d = 25,600,000, m = 1024, ~105 GB fp32
resident in HBM, 10% correlated rows) and the ResNet18-sized window with 8
fused queries. No output of the sliding step can be checked element by element
without the whole window (every coefficient depends on the full Gram matrix),
so the fp64 oracle runs for real on the host: the rows drawn on the GPU are
copied to host memory before the library touches them, the oracle forms its
own Gram matrix (oracle.dynamic.gram_accumulate over column ranges, spread
over two tests) and slides its own window. The tests of one workload share
that state and run in file order; each stays well under two minutes.

Static: the 2048-block pruning workload (d = 4,194,304, B = 2048, m = 1024).
The oracle computes the inverse diagonal of every block (a thread pool over
blocks, spread over four tests), and the library's diagonal, scores and
global keep-mask are compared with it over all d coordinates: the mask bit
for bit.
"""

import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

from gpu_common import REL_TOL, rel_l2, require_gpu
from oracle import dynamic as odyn
from oracle import mask as omask
from oracle import static as ostatic
from synth import GradientStream, get_workload

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

_S = {}


def _log(*a):
    print("[fullsize]", *a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _setup_window(dev, name, seed):
    from paper_2107_03356_amd import Window
    wl = get_workload(name)
    d, m = wl.d, wl.m
    t0 = time.perf_counter()
    gs = GradientStream(wl, seed=seed, device=dev)
    win = Window(d, m, wl.lam, max_queries=wl.queries, device=dev)
    G = np.empty((m, d), np.float32)
    batch = max(1, min(m, (2 << 30) // (4 * d)))
    for r0 in range(0, m, batch):
        n = min(batch, m - r0)
        rows = gs.rows(r0, n)
        G[r0:r0 + n] = rows.cpu().numpy()      # the oracle's copy, taken before the library sees the rows
        win.set_rows(r0, rows)
    win.rebuild()
    torch.cuda.synchronize()
    assert win.status() == 0
    _log(f"{name}: window on GPU and host in {time.perf_counter() - t0:.1f} s")
    return dict(wl=wl, gs=gs, win=win, G=G, K=np.zeros((m, m), np.float64, order="F"), cols_done=0)


def _gram_part(st, frac_end):
    """Fold the next column range of the window into the oracle's Gram, up to frac_end of d."""
    G = st["G"]
    m, d = G.shape
    j0 = st["cols_done"]
    j1 = int(round(d * frac_end))
    t0 = time.perf_counter()
    st["K"] = odyn.gram_accumulate(G, st["K"], j0, j1)
    st["cols_done"] = j1
    _log(f"oracle Gram columns [{j0}, {j1}) of {d} in {time.perf_counter() - t0:.1f} s")


def _oracle_of(st):
    wl = st["wl"]
    return odyn.WindowOracle(wl.d, wl.m, wl.lam, G0=st["G"], K=odyn.gram_symmetric(st["K"]), copy=False)


def _step_and_compare(st, t):
    wl, gs, win = st["wl"], st["gs"], st["win"]
    g = gs.step_row(t)
    X = gs.queries(t, wl.queries) if wl.queries else None
    if X is not None:
        y, Y = win.replace(g, X=X)
    else:
        y = win.replace(g)
    torch.cuda.synchronize()
    assert win.status() == 0
    t0 = time.perf_counter()
    orc = st.setdefault("orc", _oracle_of(st))
    yo = orc.slide(g.cpu().numpy())
    errs = [rel_l2(y.cpu().numpy(), yo)]
    if X is not None:
        Xh = X.cpu().numpy()
        Yo = orc.ihvp(Xh)
        errs += [rel_l2(Y[q].cpu().numpy(), Yo[q]) for q in range(wl.queries)]
    _log(f"{wl.name} step {t}: rel L2 {max(errs):.2e} (oracle {time.perf_counter() - t0:.1f} s)")
    assert max(errs) < REL_TOL, errs
    return errs


# ---------------------------------------------------------------- ResNet50-sized window
def test_resnet50_window_setup(dev):
    _S.clear()
    _S["r50"] = _setup_window(dev, "dyn_resnet50_d25.6m_m1024", seed=21)


def test_resnet50_window_oracle_gram_first_half(dev):
    if "r50" not in _S:
        pytest.skip("setup failed")
    _gram_part(_S["r50"], 0.5)


def test_resnet50_window_oracle_gram_second_half(dev):
    if "r50" not in _S:
        pytest.skip("setup failed")
    _gram_part(_S["r50"], 1.0)


def test_resnet50_window_sliding_step_matches_oracle(dev):
    if "r50" not in _S or _S["r50"]["cols_done"] < _S["r50"]["wl"].d:
        pytest.skip("setup failed")
    _step_and_compare(_S["r50"], 0)


def test_resnet50_window_known_sequence_matches_oracle(dev):
    """Three further steps as one mfac_window_replace_seq call (the fused
    pass the bench's sequence figure times), each output against the oracle."""
    st = _S.get("r50")
    if st is None or "orc" not in st:
        pytest.skip("setup failed")
    gs, win, orc = st["gs"], st["win"], st["orc"]
    Gn = torch.stack([gs.step_row(t) for t in (1, 2, 3)])
    Yn = win.replace_seq(Gn)
    torch.cuda.synchronize()
    assert win.status() == 0
    errs = []
    for i in range(3):
        t0 = time.perf_counter()
        yo = orc.slide(Gn[i].cpu().numpy())
        errs.append(rel_l2(Yn[i].cpu().numpy(), yo))
        _log(f"sequence step {i + 1}: rel L2 {errs[-1]:.2e} (oracle {time.perf_counter() - t0:.1f} s)")
    assert max(errs) < REL_TOL, errs


def test_resnet50_window_release(dev):
    _S.pop("r50", None)
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- ResNet18-sized window, 8 queries
def test_resnet18_window_setup(dev):
    _S["r18"] = _setup_window(dev, "dyn_resnet18_d11.2m_m1024_q8", seed=22)


def test_resnet18_window_oracle_gram(dev):
    if "r18" not in _S:
        pytest.skip("setup failed")
    _gram_part(_S["r18"], 1.0)


def test_resnet18_window_step_with_queries_matches_oracle(dev):
    if "r18" not in _S:
        pytest.skip("setup failed")
    _step_and_compare(_S["r18"], 0)


def test_resnet18_window_release(dev):
    _S.pop("r18", None)
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- static pruning workload
_ORACLE_PARTS = 4


def _pool_size():
    return max(1, min(16, os.cpu_count() or 1))


def test_static_pruning_full_size_setup(dev):
    """Draw G and theta on the GPU, keep the oracle's host copy, run the
    library's precompute + inverse diagonal + scores + mask: first in the fast
    mode (fp32 matrix cores, G left intact), then in the fp64 mode (which
    writes W over G)."""
    from paper_2107_03356_amd import StaticBlocks
    wl = get_workload("static_d4.19m_b2048_m1024")
    d, m, B = wl.d, wl.m, wl.block
    t0 = time.perf_counter()
    gs = GradientStream(wl, seed=23, device=dev)
    G = torch.empty((m, d), dtype=torch.float32, device=dev)
    for r in range(m):
        G[r] = gs.row(r)
    theta = gs.theta()
    Gh = G.cpu().numpy()       # the oracle's copy, taken before the library runs
    keep = d // 2
    fast = StaticBlocks(G, B, wl.lam, fp32=True)
    fdiag = fast.inv_diag(fp64=True)
    fmask, _ = fast.obs_mask(theta, keep)
    torch.cuda.synchronize()
    assert fast.status() == 0
    fdiag, fmask = fdiag.cpu().numpy(), fmask.cpu().numpy()
    fast.close()
    del fast
    torch.cuda.empty_cache()
    sb = StaticBlocks(G, B, wl.lam)
    diag = sb.inv_diag(fp64=True)
    mask, scores = sb.obs_mask(theta, keep)
    torch.cuda.synchronize()
    assert sb.status() == 0
    _log(f"static full size on GPU in {time.perf_counter() - t0:.1f} s")
    _S["st"] = dict(wl=wl, G=Gh, theta=theta.cpu().numpy(), keep=keep, diag=diag.cpu().numpy(),
                    scores=scores.cpu().numpy(), mask=mask.cpu().numpy(), fdiag=fdiag, fmask=fmask,
                    dref=np.full(d, np.nan), parts_done=0)
    sb.close()
    del G, sb
    torch.cuda.empty_cache()


@pytest.mark.parametrize("part", range(_ORACLE_PARTS))
def test_static_pruning_full_size_oracle_part(dev, part):
    """A quarter of the blocks through the oracle (oracle.static.inv_diag on
    a thread pool, one BLAS thread per block)."""
    from threadpoolctl import threadpool_limits
    st = _S.get("st")
    if st is None or st["parts_done"] != part:
        pytest.skip("setup failed")
    wl = st["wl"]
    nb = wl.d // wl.block
    per = nb // _ORACLE_PARTS
    blocks = range(part * per, nb if part + 1 == _ORACLE_PARTS else (part + 1) * per)
    B = wl.block
    t0 = time.perf_counter()

    def one(b):
        st["dref"][b * B:(b + 1) * B] = ostatic.inv_diag(st["G"], wl.lam, B, blocks=[b])

    with threadpool_limits(1), ThreadPoolExecutor(_pool_size()) as ex:
        list(ex.map(one, blocks))
    st["parts_done"] = part + 1
    _log(f"oracle blocks {blocks.start}..{blocks.stop - 1} in {time.perf_counter() - t0:.1f} s "
         f"({_pool_size()} threads)")


def test_static_pruning_full_size_matches_oracle(dev):
    """Inverse diagonal over all d coordinates (fp64, 1e-11 relative L2 and
    per block), the fp64 scores, and the global top-50% keep-mask bit for bit
    against the oracle's (Section 4.1: global OBD pruning, ties by index);
    the fast mode's keep-mask bit for bit against the same oracle mask."""
    st = _S.get("st")
    if st is None or st["parts_done"] != _ORACLE_PARTS:
        pytest.skip("oracle incomplete")
    wl, keep = st["wl"], st["keep"]
    B = wl.block
    dref = st["dref"]
    assert np.all(np.isfinite(dref))
    diag = st["diag"]
    assert rel_l2(diag, dref) < 1e-11
    blk = np.abs(diag - dref).reshape(-1, B).max(axis=1) / np.abs(dref).reshape(-1, B).max(axis=1)
    _log(f"diag: rel L2 {rel_l2(diag, dref):.2e}, worst block max rel err {blk.max():.2e} (block {blk.argmax()})")
    assert blk.max() < 1e-11
    sref = omask.scores(st["theta"], dref)
    nz = sref > 0
    srel = np.abs(st["scores"][nz] - sref[nz]) / sref[nz]
    _log(f"scores: max rel err {srel.max():.2e}")
    assert srel.max() < 1e-11
    mref = omask.keep_mask(sref, keep)
    mask = st["mask"]
    assert int(mask.sum()) == keep
    diff = np.flatnonzero(mask != mref)
    assert diff.size == 0, (diff.size, diff[:10])
    # the fast mode: fp32 rounding in its diagonal, the same mask bit for bit
    # (its band at the cut decided in fp64)
    fdiag, fmask = st["fdiag"], st["fmask"]
    frel = np.abs(fdiag - dref) / np.abs(dref)
    _log(f"fast mode: diag rel L2 {rel_l2(fdiag, dref):.2e}, max rel err {frel.max():.2e}")
    assert rel_l2(fdiag, dref) < 1e-6
    fdiff = np.flatnonzero(fmask != mref)
    assert fdiff.size == 0, (fdiff.size, fdiff[:10])


def test_static_pruning_full_size_release(dev):
    _S.pop("st", None)
