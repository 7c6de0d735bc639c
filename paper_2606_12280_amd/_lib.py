"""ctypes view of libw8a8.so, the C ABI declared in include/w8a8.h.

Loading fails loudly (ImportError-like RuntimeError) when the library has not
been built: there is no fallback implementation."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libw8a8.so")

W8A8_OK = 0
STATUS_NAMES = {
    0: "W8A8_OK", 1: "W8A8_ERR_NULL", 2: "W8A8_ERR_SHAPE", 3: "W8A8_ERR_ALIGN",
    4: "W8A8_ERR_ALIAS", 5: "W8A8_ERR_UNSUPPORTED", 6: "W8A8_ERR_HIP",
}

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_S = ctypes.c_int

# name -> (argtypes, restype), in the order of include/w8a8.h
# W8A8_MOMENTS_WORK_BYTES of the header: scratch of w8a8_act_moments.
MOMENTS_WORK_BYTES = 6 * 1024 * 8

SIGNATURES = {
    "w8a8_abi_version": ([], ctypes.c_int),
    "w8a8_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "w8a8_last_hip_error": ([], ctypes.c_char_p),
    "w8a8_act_absmax": ([_P, _I64, _I64, _P, _P], _S),
    "w8a8_act_moments": ([_P, _I64, _I64, _P, _P, _P], _S),
    "w8a8_act_moments_noalloc": ([_P, _I64, _I64, _P, _P], _S),
    "w8a8_fragility_scores": ([_P, _I64, _I64, _I64, _I64, _P], _S),
    "w8a8_select_protected": ([_P, _I64, _I64, _P], _S),
    "w8a8_rank_correlation": ([_P, _P, _I64, _P], _S),
    "w8a8_smooth_factors": ([_P, _P, _I64, _I64, ctypes.c_double, _P, _P], _S),
    "w8a8_prepare_weight": ([_P, _P, _I64, _I64, _P, _P, _P, _P], _S),
    "w8a8_quant_act": ([_P, _P, _I64, _I64, _P, _P, _P], _S),
    "w8a8_adaln_quant_act": ([_P, _P, _P, _P, _I64, _I64, ctypes.c_double, _P, _P, _P], _S),
    "w8a8_linear": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P, _P], _S),
    "w8a8_gemm_i32": ([_P, _P, _I64, _I64, _I64, _P, _P], _S),
    "bf16_linear": ([_P, _P, _P, _I64, _I64, _I64, _P, _P], _S),
    "w8a8_gemm_config": ([_I64, _I64, _I64, ctypes.c_int, _P, _P, _P], _S),
    "q8_0_quantize": ([_P, _I64, _I64, _P, _P, _P], _S),
    "q8_0_dequantize": ([_P, _P, _I64, _I64, _P, _P], _S),
    "q8_0_linear": ([_P, _P, _P, _P, _I64, _I64, _I64, _P, _P, _P], _S),
    "q4_k_quantize": ([_P, _I64, _I64, _P, _P, _P, _P, _P], _S),
    "q4_k_dequantize": ([_P, _P, _P, _P, _I64, _I64, _P, _P], _S),
    "q4_k_linear": ([_P, _P, _P, _P, _P, _P, _I64, _I64, _I64, _P, _P, _P], _S),
}

_lib = None


class W8A8Error(RuntimeError):
    """A non-zero w8a8_status returned by the library."""

    def __init__(self, fn: str, status: int, detail: str = ""):
        self.status = status
        name = STATUS_NAMES.get(status, str(status))
        msg = f"{fn}: {name}"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


def load():
    """Load libw8a8.so once and declare every entry point's signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2606_12280_amd.build` "
            "(the W8A8 path has no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (args, res) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def check(fn: str, status: int) -> None:
    if status != W8A8_OK:
        lib = load()
        detail = lib.w8a8_status_string(status).decode()
        if status == 6:
            detail += ": " + lib.w8a8_last_hip_error().decode()
        raise W8A8Error(fn, status, detail)
