"""MI355X-native fused multi-table embedding lookup (DPIFrame's embedding hot path).

The compute path is libdpi.so (HIP for gfx950) behind the C ABI in
include/dpi.h; this package is its Python binding.
"""
from . import dpi  # noqa: F401
from .dpi import DpiError, load  # noqa: F401
