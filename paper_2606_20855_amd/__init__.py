"""MI355X (gfx950) SpGEMM: C = A * B with CSR inputs and a CSR output.

The computation lives in libwingspan.so (hand-written HIP kernels behind the
C ABI of include/wingspan.h); `wingspan` is its Python binding.
"""
from . import wingspan
from .wingspan import DeviceCSR, WingspanError, spgemm

__all__ = ["wingspan", "DeviceCSR", "WingspanError", "spgemm"]
