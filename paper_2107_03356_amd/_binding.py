"""ctypes binding of libmfac (include/mfac.h), argument marshalling only.

Every public C function has a Python function of the same name taking plain
integers (device pointers, sizes, stream handles) and returning the status
code. ``Window`` and ``StaticBlocks`` are thin owners of the caller-side
buffers (allocated with torch, which is used only for device memory and
streams) that call those functions and raise ``MfacError`` on a non-zero
status. There is no fallback: if libmfac.so is missing, loading fails loudly.
"""

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmfac.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "mfac.h")

MFAC_OK = 0
MFAC_EINVAL = -1
MFAC_EWORKSPACE = -2
MFAC_EHIP = -3
MFAC_ENONFINITE = -4
MFAC_ESTATE = -5
MFAC_EPRECISION = -6
MFAC_STATIC_TRACE = 1
MFAC_STATIC_FP32 = 2

_c = ctypes
_VP, _I32, _I64, _SZ, _F32, _F64 = _c.c_void_p, _c.c_int32, _c.c_int64, _c.c_size_t, _c.c_float, _c.c_double
_PVP = _c.POINTER(_c.c_void_p)

# name -> (restype, argtypes)
SIGNATURES = {
    "mfac_status_string": (_c.c_char_p, [_c.c_int]),
    "mfac_version": (_I32, []),
    "mfac_window_storage_bytes": (_SZ, [_I64, _I32]),
    "mfac_window_workspace_bytes": (_SZ, [_I64, _I32, _I32]),
    "mfac_window_init": (_c.c_int, [_PVP, _I64, _I32, _F64, _I32, _VP, _SZ, _VP, _SZ, _VP, _VP]),
    "mfac_window_set_rows": (_c.c_int, [_VP, _I32, _I32, _VP]),
    "mfac_window_rebuild": (_c.c_int, [_VP]),
    "mfac_window_replace": (_c.c_int, [_VP, _I32, _VP, _VP, _I32, _VP, _VP]),
    "mfac_window_replace_seq": (_c.c_int, [_VP, _I32, _VP, _VP]),
    "mfac_ihvp": (_c.c_int, [_VP, _I32, _VP, _VP]),
    "mfac_ihvp_noalloc": (_c.c_int, [_VP, _I32, _VP, _VP]),
    "mfac_window_get_rows": (_c.c_int, [_VP, _I32, _I32, _VP]),
    "mfac_window_info": (_c.c_int, [_VP, _c.POINTER(_I32), _c.POINTER(_I64)]),
    "mfac_window_set_head": (_c.c_int, [_VP, _I32, _I64]),
    "mfac_window_set_refactor_period": (_c.c_int, [_VP, _I32]),
    "mfac_window_set_stream": (_c.c_int, [_VP, _VP]),
    "mfac_window_trace": (_c.c_int, [_VP, _I32]),
    "mfac_window_trace_read": (_c.c_int, [_VP, _c.POINTER(_F64), _c.POINTER(_I64)]),
    "mfac_window_status": (_c.c_int, [_VP]),
    "mfac_window_destroy": (_c.c_int, [_VP]),
    "mfac_static_workspace_bytes": (_SZ, [_I64, _I32, _I32]),
    "mfac_static_workspace_bytes_flags": (_SZ, [_I64, _I32, _I32, _c.c_uint32]),
    "mfac_static_precompute": (_c.c_int, [_PVP, _I64, _I32, _I32, _F64, _VP, _VP, _SZ, _c.c_uint32, _VP]),
    "mfac_static_paged_workspace_bytes": (_SZ, [_I64, _I32, _I32, _I64]),
    "mfac_static_precompute_paged": (_c.c_int, [_PVP, _I64, _I32, _I32, _F64, _VP, _I64, _VP, _SZ, _c.c_uint32,
                                                _VP]),
    "mfac_static_trace_read": (_c.c_int, [_VP, _c.POINTER(_F64), _c.POINTER(_I64)]),
    "mfac_inv_diag": (_c.c_int, [_VP, _VP]),
    "mfac_inv_diag64": (_c.c_int, [_VP, _VP]),
    "mfac_obs_mask": (_c.c_int, [_VP, _VP, _I64, _VP, _VP]),
    "mfac_static_ihvp": (_c.c_int, [_VP, _I32, _VP, _VP]),
    "mfac_static_element": (_c.c_int, [_VP, _I64, _VP, _VP]),
    "mfac_obs_update": (_c.c_int, [_VP, _VP, _VP, _VP]),
    "mfac_static_set_stream": (_c.c_int, [_VP, _VP]),
    "mfac_static_status": (_c.c_int, [_VP]),
    "mfac_static_destroy": (_c.c_int, [_VP]),
}

_lib = None


class MfacError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({status_string(status)})")


def header_symbols(path=HEADER):
    """Names of the functions declared in include/mfac.h."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mfac_[a-z0-9_]+)\s*\(", text)))


def load(path=LIB_PATH):
    """Load libmfac.so (built in place by paper_2107_03356_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libmfac.so not found at {path}: run `python -m paper_2107_03356_amd.build` first")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_string(status):
    return load().mfac_status_string(int(status)).decode()


def _check(fn, status):
    if status != MFAC_OK:
        raise MfacError(fn, status)


# ---------------------------------------------------------------- same-name calls
def _mk(name):
    def call(*args):
        return getattr(load(), name)(*args)
    call.__name__ = name
    return call


for _n in SIGNATURES:
    globals()[_n] = _mk(_n)


# ---------------------------------------------------------------- buffer owners
def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream_handle(torch, device, stream):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


class Window:
    """A sliding window of m gradients of dimension d on one GPU.

    Owns the window storage and workspace (torch uint8 buffers) and the C
    handle. ``replace`` is the optimizer step (Section 4.2), ``ihvp`` the
    plain IHVP.
    """

    def __init__(self, d, m, lam, max_queries=0, G0=None, device="cuda", stream=None):
        import torch
        self.torch = torch
        self.d, self.m, self.lam, self.max_queries = int(d), int(m), float(lam), int(max_queries)
        self.device = torch.device(device)
        lib = load()
        sb = lib.mfac_window_storage_bytes(self.d, self.m)
        wb = lib.mfac_window_workspace_bytes(self.d, self.m, self.max_queries)
        if sb == 0 or wb == 0:
            raise MfacError("mfac_window_workspace_bytes", MFAC_EINVAL)
        self.storage = torch.empty(sb, dtype=torch.uint8, device=self.device)
        self.workspace = torch.empty(wb, dtype=torch.uint8, device=self.device)
        if G0 is not None:
            assert G0.dtype == torch.float32 and G0.is_contiguous() and G0.shape == (self.m, self.d)
        self.stream = _stream_handle(torch, self.device, stream)
        h = ctypes.c_void_p()
        st = lib.mfac_window_init(ctypes.byref(h), self.d, self.m, self.lam, self.max_queries,
                                  _ptr(self.storage), sb, _ptr(self.workspace), wb, _ptr(G0), self.stream)
        _check("mfac_window_init", st)
        self.handle = h

    def _vec(self, x, n=None):
        t = self.torch
        assert x.dtype == t.float32 and x.is_contiguous() and x.device == self.device
        if n is not None:
            assert x.numel() == n * self.d
        return x

    def replace(self, g, slot=-1, y_out=None, X=None, Y=None, want_y=True):
        """Insert g (into ``slot``, or the ring head) and return F^-1 g."""
        t = self.torch
        self._vec(g, 1)
        if want_y and y_out is None:
            y_out = t.empty(self.d, dtype=t.float32, device=self.device)
        n = 0
        if X is not None:
            n = X.shape[0] if X.dim() == 2 else 1
            self._vec(X, n)
            if Y is None:
                Y = t.empty_like(X)
            self._vec(Y, n)
        st = load().mfac_window_replace(self.handle, int(slot), _ptr(g), _ptr(y_out), n, _ptr(X), _ptr(Y))
        _check("mfac_window_replace", st)
        return (y_out, Y) if X is not None else y_out

    def replace_seq(self, Gn, Yn=None):
        """Insert the rows of Gn (n x d) one after another into the ring head;
        row t of the result is F^-1 Gn[t] right after Gn[t] went in."""
        t = self.torch
        n = Gn.shape[0]
        self._vec(Gn, n)
        if Yn is None:
            Yn = t.empty_like(Gn)
        self._vec(Yn, n)
        _check("mfac_window_replace_seq", load().mfac_window_replace_seq(self.handle, n, _ptr(Gn), _ptr(Yn)))
        return Yn

    def ihvp(self, X, Y=None):
        t = self.torch
        n = X.shape[0] if X.dim() == 2 else 1
        self._vec(X, n)
        if Y is None:
            Y = t.empty_like(X)
        _check("mfac_ihvp", load().mfac_ihvp(self.handle, n, _ptr(X), _ptr(Y)))
        return Y

    def set_rows(self, first, rows):
        self._vec(rows, rows.shape[0])
        _check("mfac_window_set_rows", load().mfac_window_set_rows(self.handle, int(first), rows.shape[0], _ptr(rows)))

    def rebuild(self):
        _check("mfac_window_rebuild", load().mfac_window_rebuild(self.handle))

    def get_rows(self, first=0, count=None):
        t = self.torch
        count = self.m - first if count is None else count
        out = t.empty((count, self.d), dtype=t.float32, device=self.device)
        _check("mfac_window_get_rows", load().mfac_window_get_rows(self.handle, int(first), int(count), _ptr(out)))
        return out

    def info(self):
        h, s = ctypes.c_int32(), ctypes.c_int64()
        _check("mfac_window_info", load().mfac_window_info(self.handle, ctypes.byref(h), ctypes.byref(s)))
        return h.value, s.value

    def set_head(self, head, steps):
        _check("mfac_window_set_head", load().mfac_window_set_head(self.handle, int(head), int(steps)))

    def set_stream(self, stream=None):
        """Bind later calls to ``stream`` (a torch stream; default: the current
        one). The new stream first waits for the work already enqueued on the
        old one, so the window's calls stay in order across the switch."""
        t = self.torch
        new = stream if stream is not None else t.cuda.current_stream(self.device)
        if new.cuda_stream == self.stream:
            return
        ev = t.cuda.Event()
        ev.record(t.cuda.ExternalStream(self.stream, device=self.device))
        new.wait_event(ev)
        self.stream = new.cuda_stream
        _check("mfac_window_set_stream", load().mfac_window_set_stream(self.handle, self.stream))

    def set_refactor_period(self, period):
        _check("mfac_window_set_refactor_period", load().mfac_window_set_refactor_period(self.handle, int(period)))

    def trace(self, enable=True):
        _check("mfac_window_trace", load().mfac_window_trace(self.handle, 1 if enable else 0))

    def trace_read(self):
        """(ms per phase, launches per phase) since the last read; phases: pass 1,
        coefficients, pass 2, row write."""
        ms = (ctypes.c_double * 4)()
        cnt = (ctypes.c_int64 * 4)()
        _check("mfac_window_trace_read", load().mfac_window_trace_read(self.handle, ms, cnt))
        return list(ms), list(cnt)

    def status(self):
        return load().mfac_window_status(self.handle)

    def close(self):
        if getattr(self, "handle", None) is not None:
            load().mfac_window_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class StaticBlocks:
    """Static block-wise precompute over a caller's m x d gradient matrix.

    G is overwritten in place by W (W_b = R_b^-1 G_b per block), except with
    ``fp32=True`` (the fast mode: fp32 matrix cores, G left intact, W formed in
    the workspace by the first query, the keep-mask still exact). G is either a
    device tensor, or (``page_cols`` given) a pinned host tensor
    (``pin_memory=True``) larger than the device should hold: it then passes
    through the device in pages of ``page_cols`` columns (whole blocks when
    block < d), and the queries read W from host memory.
    """

    def __init__(self, G, block, lam, stream=None, trace=False, page_cols=None, device=None, fp32=False):
        import torch
        self.torch = torch
        assert G.dtype == torch.float32 and G.is_contiguous() and G.dim() == 2
        self.G = G
        self.m, self.d = G.shape
        self.block, self.lam = int(block), float(lam)
        lib = load()
        flags = (MFAC_STATIC_TRACE if trace else 0) | (MFAC_STATIC_FP32 if fp32 else 0)
        h = ctypes.c_void_p()
        if page_cols is None:
            self.device = G.device
            wb = lib.mfac_static_workspace_bytes_flags(self.d, self.block, self.m, flags)
            if wb == 0:
                raise MfacError("mfac_static_workspace_bytes_flags", MFAC_EINVAL)
            self.workspace = torch.empty(wb, dtype=torch.uint8, device=self.device)
            self.stream = _stream_handle(torch, self.device, stream)
            st = lib.mfac_static_precompute(ctypes.byref(h), self.d, self.block, self.m, self.lam, _ptr(G),
                                            _ptr(self.workspace), wb, flags, self.stream)
            _check("mfac_static_precompute", st)
        else:
            if G.device.type != "cpu" or not G.is_pinned():
                raise ValueError("StaticBlocks: a paged G must be a pinned host tensor (pin_memory=True)")
            self.device = torch.device(device if device is not None else "cuda")
            wb = lib.mfac_static_paged_workspace_bytes(self.d, self.block, self.m, int(page_cols))
            if wb == 0:
                raise MfacError("mfac_static_paged_workspace_bytes", MFAC_EINVAL)
            self.workspace = torch.empty(wb, dtype=torch.uint8, device=self.device)
            self.stream = _stream_handle(torch, self.device, stream)
            st = lib.mfac_static_precompute_paged(ctypes.byref(h), self.d, self.block, self.m, self.lam, _ptr(G),
                                                  int(page_cols), _ptr(self.workspace), wb, flags, self.stream)
            _check("mfac_static_precompute_paged", st)
        self.handle = h

    def trace_read(self):
        """(ms per stage, launches per stage) since creation or the last read;
        stages: Gram, factor and inverse, W and diagonal, scores and mask.
        Zeros unless created with trace=True."""
        ms = (ctypes.c_double * 4)()
        cnt = (ctypes.c_int64 * 4)()
        _check("mfac_static_trace_read", load().mfac_static_trace_read(self.handle, ms, cnt))
        return list(ms), list(cnt)

    def inv_diag(self, out=None, fp64=False):
        t = self.torch
        if fp64:
            out = t.empty(self.d, dtype=t.float64, device=self.device) if out is None else out
            _check("mfac_inv_diag64", load().mfac_inv_diag64(self.handle, _ptr(out)))
        else:
            out = t.empty(self.d, dtype=t.float32, device=self.device) if out is None else out
            _check("mfac_inv_diag", load().mfac_inv_diag(self.handle, _ptr(out)))
        return out

    def obs_mask(self, theta, keep, scores=True):
        t = self.torch
        assert theta.dtype == t.float32 and theta.numel() == self.d
        sc = t.empty(self.d, dtype=t.float64, device=self.device) if scores else None
        mask = t.empty(self.d, dtype=t.uint8, device=self.device)
        _check("mfac_obs_mask", load().mfac_obs_mask(self.handle, _ptr(theta), int(keep), _ptr(sc), _ptr(mask)))
        return mask, sc

    def ihvp(self, X, Y=None):
        """F^-1 X for the block-wise Fisher (n <= 4 rows of length d)."""
        t = self.torch
        n = X.shape[0] if X.dim() == 2 else 1
        assert X.dtype == t.float32 and X.is_contiguous() and X.numel() == n * self.d
        Y = t.empty_like(X) if Y is None else Y
        _check("mfac_static_ihvp", load().mfac_static_ihvp(self.handle, n, _ptr(X), _ptr(Y)))
        return Y

    def element(self, ij):
        """[F^-1]_ij for an (nq, 2) int64 tensor of index pairs; returns nq fp64."""
        t = self.torch
        ij = ij.to(device=self.device, dtype=t.int64).contiguous()
        out = t.empty(ij.shape[0], dtype=t.float64, device=self.device)
        _check("mfac_static_element", load().mfac_static_element(self.handle, ij.shape[0], _ptr(ij), _ptr(out)))
        return out

    def obs_update(self, theta, keep_mask, delta=None):
        """OBS correction delta (fp32, d) for removing the coordinates outside keep_mask."""
        t = self.torch
        assert theta.dtype == t.float32 and keep_mask.dtype == t.uint8
        if delta is None:
            delta = t.empty(self.d, dtype=t.float32, device=self.device)
        assert delta.dtype == t.float32 and delta.is_contiguous() and delta.numel() == self.d
        _check("mfac_obs_update", load().mfac_obs_update(self.handle, _ptr(theta), _ptr(keep_mask), _ptr(delta)))
        return delta

    def status(self):
        return load().mfac_static_status(self.handle)

    def close(self):
        if getattr(self, "handle", None) is not None:
            load().mfac_static_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
