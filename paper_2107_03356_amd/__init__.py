"""MI355X-native M-FAC inverse-Hessian-vector products (gfx950 HIP kernels).

The library is libmfac.so (C ABI in include/mfac.h), built in place by
``python -m paper_2107_03356_amd.build``. This package is its Python binding.
"""

from ._binding import (  # noqa: F401
    MFAC_EHIP,
    MFAC_EINVAL,
    MFAC_EPRECISION,
    MFAC_ENONFINITE,
    MFAC_ESTATE,
    MFAC_EWORKSPACE,
    MFAC_OK,
    LIB_PATH,
    MfacError,
    StaticBlocks,
    Window,
    header_symbols,
    load,
    status_string,
)
from . import _binding as capi  # noqa: F401  (same-name C calls: capi.mfac_window_init, ...)
