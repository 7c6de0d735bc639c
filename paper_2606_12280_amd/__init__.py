"""MI355X (gfx950) INT8 W8A8 quantized linear: SmoothQuant smoothing,
per-token dynamic INT8 activations, per-channel INT8 weights, an INT8 MFMA
GEMM with a fused dequantization epilogue, and a bf16 path for protected
layers (arXiv 2606.12280, Section 3).

The compute lives in libw8a8.so (C ABI: include/w8a8.h); ``ops`` is its torch
binding and ``layer`` the per-layer routing."""
from . import layer, ops  # noqa: F401
from ._lib import LIB_PATH, W8A8Error, load  # noqa: F401
