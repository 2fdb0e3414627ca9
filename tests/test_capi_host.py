"""The C ABI on the host: the library loads, exports every declared symbol, and
rejects bad arguments before touching the device (no GPU needed)."""

import ctypes
import os

import pytest

from paper_2107_03356_amd import _binding as B

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIB_PATH), reason="libmfac.so not built")


def test_exports_every_header_symbol():
    lib = B.load()
    names = B.header_symbols()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(B.SIGNATURES), set(names) ^ set(B.SIGNATURES)


def test_status_strings_and_version():
    assert B.status_string(B.MFAC_OK) == "ok"
    assert "invalid" in B.status_string(B.MFAC_EINVAL)
    assert B.load().mfac_version() >= 100


def test_size_queries():
    lib = B.load()
    # slab layout: columns rounded up to 2048 per slab
    assert lib.mfac_window_storage_bytes(4096, 16) == 4096 * 16 * 4
    assert lib.mfac_window_storage_bytes(4097, 16) == 3 * 2048 * 16 * 4
    assert lib.mfac_window_storage_bytes(0, 16) == 0
    assert lib.mfac_window_workspace_bytes(4096, 16, 0) > 0
    assert lib.mfac_window_workspace_bytes(4096, 16, 17) == 0     # too many queries
    assert lib.mfac_window_workspace_bytes(4096, 0, 0) == 0
    assert lib.mfac_window_workspace_bytes(4096, 16384, 1) == 0   # m * (q + 1) too large
    assert lib.mfac_static_workspace_bytes(4096, 256, 64) > 4096 * 16
    assert lib.mfac_static_workspace_bytes(4096, 300, 64) == 0    # block does not divide d
    assert lib.mfac_static_workspace_bytes(4096, 2, 64) == 0      # block not a multiple of 4


def _init(**kw):
    lib = B.load()
    a = dict(d=4096, m=16, lam=1e-3, q=0, storage=256 * 1000, sb=1 << 30, ws=256 * 2000, wb=1 << 30, G0=None)
    a.update(kw)
    h = ctypes.c_void_p()
    return lib.mfac_window_init(ctypes.byref(h), a["d"], a["m"], a["lam"], a["q"], a["storage"], a["sb"],
                                a["ws"], a["wb"], a["G0"], None), h


@pytest.mark.parametrize("kw,expect", [
    (dict(m=0), B.MFAC_EINVAL),
    (dict(d=0), B.MFAC_EINVAL),
    (dict(lam=0.0), B.MFAC_EINVAL),
    (dict(lam=-1.0), B.MFAC_EINVAL),
    (dict(lam=float("nan")), B.MFAC_EINVAL),
    (dict(lam=float("inf")), B.MFAC_EINVAL),
    (dict(q=17), B.MFAC_EINVAL),
    (dict(d=(1 << 34) + 4), B.MFAC_EINVAL),          # past the 32-bit work-item count of d/4 launches
    (dict(storage=None), B.MFAC_EINVAL),
    (dict(ws=None), B.MFAC_EINVAL),
    (dict(storage=256 * 1000 + 4), B.MFAC_EINVAL),     # not 256-byte aligned
    (dict(G0=256 * 3 + 2), B.MFAC_EINVAL),             # misaligned initial rows
    (dict(sb=100), B.MFAC_EWORKSPACE),
    (dict(wb=100), B.MFAC_EWORKSPACE),
])
def test_window_init_rejects_on_host(kw, expect):
    st, h = _init(**kw)
    assert st == expect
    assert h.value is None


def test_null_handles_and_out_pointers():
    lib = B.load()
    assert lib.mfac_window_init(None, 4096, 16, 1e-3, 0, 256, 1 << 30, 512, 1 << 30, None, None) == B.MFAC_EINVAL
    assert lib.mfac_window_replace(None, -1, 256, 512, 0, None, None) == B.MFAC_EINVAL
    assert lib.mfac_window_replace_seq(None, 2, 256, 512) == B.MFAC_EINVAL
    assert lib.mfac_ihvp(None, 1, 256, 512) == B.MFAC_EINVAL
    assert lib.mfac_window_rebuild(None) == B.MFAC_EINVAL
    assert lib.mfac_window_status(None) == B.MFAC_EINVAL
    assert lib.mfac_window_set_rows(None, 0, 1, 256) == B.MFAC_EINVAL
    assert lib.mfac_window_get_rows(None, 0, 1, 256) == B.MFAC_EINVAL
    assert lib.mfac_window_info(None, None, None) == B.MFAC_EINVAL
    assert lib.mfac_window_destroy(None) == B.MFAC_OK
    assert lib.mfac_inv_diag(None, 256) == B.MFAC_EINVAL
    assert lib.mfac_obs_mask(None, 256, 1, None, 512) == B.MFAC_EINVAL
    assert lib.mfac_static_destroy(None) == B.MFAC_OK


@pytest.mark.parametrize("args,expect", [
    ((4096, 300, 64, 1e-4), B.MFAC_EINVAL),   # d % block != 0
    ((4096, 256, 0, 1e-4), B.MFAC_EINVAL),
    ((4096, 256, 64, 0.0), B.MFAC_EINVAL),
    ((4096, 256, 64, float("nan")), B.MFAC_EINVAL),
    (((1 << 32), 1 << 20, 64, 1e-4), B.MFAC_EINVAL),   # d past 2^32 - 256 (one work-item per coordinate)
])
def test_static_precompute_rejects_on_host(args, expect):
    lib = B.load()
    h = ctypes.c_void_p()
    d, blk, m, lam = args
    assert lib.mfac_static_precompute(ctypes.byref(h), d, blk, m, lam, 256, 512, 1 << 40, 0, None) == expect
    assert h.value is None
    # workspace too small
    assert lib.mfac_static_precompute(ctypes.byref(h), 4096, 256, 64, 1e-4, 256, 512, 16, 0, None) == B.MFAC_EWORKSPACE
    # unknown flag bits
    assert lib.mfac_static_precompute(ctypes.byref(h), 4096, 256, 64, 1e-4, 256, 512, 1 << 40, 6,
                                      None) == B.MFAC_EINVAL


def test_trace_read_rejects_null_arguments():
    lib = B.load()
    ms = (ctypes.c_double * 4)()
    cnt = (ctypes.c_int64 * 4)()
    assert lib.mfac_static_trace_read(None, ms, cnt) == B.MFAC_EINVAL
    assert lib.mfac_window_trace_read(None, ms, cnt) == B.MFAC_EINVAL


def test_paged_plan_validation_on_host():
    lib = B.load()
    ws = lib.mfac_static_paged_workspace_bytes
    assert ws(4096, 256, 64, 1024) > 0
    assert ws(4096, 256, 64, 2048) > ws(4096, 256, 64, 1024)     # two bigger page buffers, more blocks per page
    assert ws(4096, 256, 64, 1000) == 0      # not whole blocks
    assert ws(4096, 256, 64, 2) == 0         # below 4 columns
    assert ws(4096, 4096, 64, 1026) == 0     # full-d pages: a multiple of 4
    assert ws(4096, 4096, 64, 1024) > 0
    assert ws(4096, 4096, 64, 1 << 20) == ws(4096, 4096, 64, 4096)   # pages wider than d mean d
    h = ctypes.c_void_p()
    for page in (1000, 2, 0):
        assert lib.mfac_static_precompute_paged(ctypes.byref(h), 4096, 256, 64, 1e-4, 256, page, 512, 1 << 40, 0,
                                                None) == B.MFAC_EINVAL
        assert h.value is None
    assert lib.mfac_static_precompute_paged(None, 4096, 256, 64, 1e-4, 256, 1024, 512, 1 << 40, 0,
                                            None) == B.MFAC_EINVAL
