"""Torch-tensor binding of the C ABI (include/w8a8.h), same names.

Argument marshalling only: each function checks dtypes, devices and
contiguity, allocates missing outputs with torch (device memory is all torch
provides here), passes raw device pointers and torch's current HIP stream to
the library, and raises W8A8Error on a non-zero status. Every arithmetic step
runs in the library's HIP kernels. bf16 tensors are torch.bfloat16."""
from __future__ import annotations

import ctypes

import torch

from ._lib import MOMENTS_WORK_BYTES, check, load

__all__ = [
    "w8a8_act_absmax", "w8a8_smooth_factors", "w8a8_prepare_weight", "w8a8_quant_act",
    "w8a8_linear", "w8a8_gemm_i32", "bf16_linear",
]


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, ndim: int, device=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got shape {tuple(t.shape)}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU, got {t.device}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _need_vec(t: torch.Tensor, name: str, dtype: torch.dtype, n: int, device=None) -> torch.Tensor:
    """A 1-D operand of exactly n entries: the C ABI takes no lengths, so a
    shorter vector would be read past its end."""
    _need(t, name, dtype, 1, device)
    if t.numel() != n:
        raise ValueError(f"{name} must have {n} entries, got {t.numel()}")
    return t


def _out(t, shape, dtype, device, name):
    if t is None:
        return torch.empty(shape, dtype=dtype, device=device)
    _need(t, name, dtype, len(shape), device)
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def w8a8_act_absmax(X: torch.Tensor, absmax: torch.Tensor) -> torch.Tensor:
    """absmax[k] = max(absmax[k], max_t |X[t, k]|), in place (calibration)."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    _need_vec(absmax, "absmax", torch.float32, K, X.device)
    lib = load()
    with torch.cuda.device(X.device):
        check("w8a8_act_absmax",
              lib.w8a8_act_absmax(_ptr(X), M, K, _ptr(absmax), _stream(X.device)))
    return absmax


def w8a8_act_moments(X: torch.Tensor, work: torch.Tensor | None = None,
                     out: torch.Tensor | None = None) -> torch.Tensor:
    """Fragility statistics of a linear's input: float64 [max |x|, mean,
    population std, Pearson kurtosis] on X's device. `work` (uint8, at least
    MOMENTS_WORK_BYTES) may be passed to avoid allocating it per call."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    stats = _out(out, (4,), torch.float64, X.device, "out")
    if work is None:
        work = torch.empty(MOMENTS_WORK_BYTES, dtype=torch.uint8, device=X.device)
    _need(work, "work", torch.uint8, 1, X.device)
    if work.numel() < MOMENTS_WORK_BYTES:
        raise ValueError(f"work needs {MOMENTS_WORK_BYTES} bytes")
    lib = load()
    with torch.cuda.device(X.device):
        check("w8a8_act_moments",
              lib.w8a8_act_moments(_ptr(X), M, K, _ptr(work), _ptr(stats), _stream(X.device)))
    return stats


def w8a8_act_moments_noalloc(X: torch.Tensor, out: torch.Tensor) -> torch.Tensor:
    """w8a8_act_moments with no workspace: the library's own device array
    holds the partial states (for callers that cannot allocate; `out`, float64
    [4] on X's device, is required). Calls that overlap on one GPU race."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    stats = _out(out, (4,), torch.float64, X.device, "out")
    lib = load()
    with torch.cuda.device(X.device):
        check("w8a8_act_moments_noalloc",
              lib.w8a8_act_moments_noalloc(_ptr(X), M, K, _ptr(stats), _stream(X.device)))
    return stats


def w8a8_smooth_factors(act_absmax: torch.Tensor, W: torch.Tensor, alpha: float = 0.5,
                        out: torch.Tensor | None = None) -> torch.Tensor:
    """lambda_j = s_j^alpha / max_i |W_ij|^(1 - alpha) -> fp32 [K]."""
    _need(W, "W", torch.bfloat16, 2)
    N, K = W.shape
    _need_vec(act_absmax, "act_absmax", torch.float32, K, W.device)
    lam = _out(out, (K,), torch.float32, W.device, "out")
    lib = load()
    with torch.cuda.device(W.device):
        check("w8a8_smooth_factors",
              lib.w8a8_smooth_factors(_ptr(act_absmax), _ptr(W), N, K, float(alpha), _ptr(lam),
                                      _stream(W.device)))
    return lam


def w8a8_prepare_weight(W: torch.Tensor, lam: torch.Tensor, Wq=None, w_scale=None,
                        inv_lambda=None):
    """Offline weight side -> (Wq int8 [N, K], w_scale fp32 [N], inv_lambda fp32 [K])."""
    _need(W, "W", torch.bfloat16, 2)
    N, K = W.shape
    _need_vec(lam, "lambda", torch.float32, K, W.device)
    dev = W.device
    Wq = _out(Wq, (N, K), torch.int8, dev, "Wq")
    w_scale = _out(w_scale, (N,), torch.float32, dev, "w_scale")
    inv_lambda = _out(inv_lambda, (K,), torch.float32, dev, "inv_lambda")
    lib = load()
    with torch.cuda.device(dev):
        check("w8a8_prepare_weight",
              lib.w8a8_prepare_weight(_ptr(W), _ptr(lam), N, K, _ptr(Wq), _ptr(w_scale),
                                      _ptr(inv_lambda), _stream(dev)))
    return Wq, w_scale, inv_lambda


def w8a8_quant_act(X: torch.Tensor, inv_lambda: torch.Tensor, Xq=None, x_scale=None):
    """Smooth + per-token quantize -> (Xq int8 [M, K], x_scale fp32 [M])."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    _need_vec(inv_lambda, "inv_lambda", torch.float32, K, X.device)
    dev = X.device
    Xq = _out(Xq, (M, K), torch.int8, dev, "Xq")
    x_scale = _out(x_scale, (M,), torch.float32, dev, "x_scale")
    lib = load()
    with torch.cuda.device(dev):
        check("w8a8_quant_act",
              lib.w8a8_quant_act(_ptr(X), _ptr(inv_lambda), M, K, _ptr(Xq), _ptr(x_scale),
                                 _stream(dev)))
    return Xq, x_scale


def w8a8_adaln_quant_act(X: torch.Tensor, shift: torch.Tensor, scale: torch.Tensor,
                         inv_lambda: torch.Tensor, eps: float = 1e-6, Xq=None, x_scale=None):
    """adaLN modulation (LayerNorm(X) * (1 + scale) + shift, rounded to bf16)
    fused with smooth + per-token quantize -> (Xq int8 [M, K], x_scale fp32 [M])."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    dev = X.device
    for name, t in (("shift", shift), ("scale", scale)):
        _need_vec(t, name, torch.bfloat16, K, dev)
    _need_vec(inv_lambda, "inv_lambda", torch.float32, K, dev)
    Xq = _out(Xq, (M, K), torch.int8, dev, "Xq")
    x_scale = _out(x_scale, (M,), torch.float32, dev, "x_scale")
    lib = load()
    with torch.cuda.device(dev):
        check("w8a8_adaln_quant_act",
              lib.w8a8_adaln_quant_act(_ptr(X), _ptr(shift), _ptr(scale), _ptr(inv_lambda), M, K,
                                       float(eps), _ptr(Xq), _ptr(x_scale), _stream(dev)))
    return Xq, x_scale


def w8a8_linear(Xq: torch.Tensor, x_scale: torch.Tensor, Wq: torch.Tensor,
                w_scale: torch.Tensor, bias: torch.Tensor | None = None,
                out: torch.Tensor | None = None) -> torch.Tensor:
    """INT8 GEMM + fused dequant/bias epilogue -> Y bf16 [M, N]."""
    _need(Xq, "Xq", torch.int8, 2)
    _need(Wq, "Wq", torch.int8, 2, Xq.device)
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq must share K")
    _need_vec(x_scale, "x_scale", torch.float32, M, Xq.device)
    _need_vec(w_scale, "w_scale", torch.float32, N, Xq.device)
    if bias is not None:
        _need_vec(bias, "bias", torch.bfloat16, N, Xq.device)
    Y = _out(out, (M, N), torch.bfloat16, Xq.device, "out")
    lib = load()
    with torch.cuda.device(Xq.device):
        check("w8a8_linear",
              lib.w8a8_linear(_ptr(Xq), _ptr(x_scale), _ptr(Wq), _ptr(w_scale), _ptr(bias),
                              M, N, K, _ptr(Y), _stream(Xq.device)))
    return Y


def w8a8_gemm_i32(Xq: torch.Tensor, Wq: torch.Tensor, out: torch.Tensor | None = None):
    """The same GEMM storing the int32 accumulators -> C int32 [M, N]."""
    _need(Xq, "Xq", torch.int8, 2)
    _need(Wq, "Wq", torch.int8, 2, Xq.device)
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq must share K")
    C = _out(out, (M, N), torch.int32, Xq.device, "out")
    lib = load()
    with torch.cuda.device(Xq.device):
        check("w8a8_gemm_i32",
              lib.w8a8_gemm_i32(_ptr(Xq), _ptr(Wq), M, N, K, _ptr(C), _stream(Xq.device)))
    return C


def bf16_linear(X: torch.Tensor, W: torch.Tensor, bias: torch.Tensor | None = None,
                out: torch.Tensor | None = None) -> torch.Tensor:
    """Protected layer: bf16 X W^T + bias with fp32 accumulation -> Y bf16 [M, N]."""
    _need(X, "X", torch.bfloat16, 2)
    _need(W, "W", torch.bfloat16, 2, X.device)
    M, K = X.shape
    N = W.shape[0]
    if W.shape[1] != K:
        raise ValueError("X and W must share K")
    if bias is not None:
        _need_vec(bias, "bias", torch.bfloat16, N, X.device)
    Y = _out(out, (M, N), torch.bfloat16, X.device, "out")
    lib = load()
    with torch.cuda.device(X.device):
        check("bf16_linear",
              lib.bf16_linear(_ptr(X), _ptr(W), _ptr(bias), M, N, K, _ptr(Y), _stream(X.device)))
    return Y


def w8a8_gemm_config(M: int, N: int, K: int, bf16: bool = False) -> tuple[int, int, int]:
    """(tile_m, tile_n, threads) of the GEMM that w8a8_linear / w8a8_gemm_i32
    (bf16=False) or bf16_linear (bf16=True) launch for M x N x K. Host only."""
    tm, tn, nt = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    check("w8a8_gemm_config", load().w8a8_gemm_config(M, N, K, int(bool(bf16)), ctypes.byref(tm),
                                                      ctypes.byref(tn), ctypes.byref(nt)))
    return tm.value, tn.value, nt.value


# --------------------------------------------------------------------------
# GGUF Q8_0 weight-only
# --------------------------------------------------------------------------

Q8_0_BLOCK = 32


def q8_0_quantize(W: torch.Tensor) -> tuple[torch.Tensor, torch.Tensor]:
    """W [N, K] bf16 -> (codes int8 [N, K], scales float16 [N, K/32])."""
    _need(W, "W", torch.bfloat16, 2)
    N, K = W.shape
    qs = torch.empty(N, K, dtype=torch.int8, device=W.device)
    d = torch.empty(N, K // Q8_0_BLOCK, dtype=torch.float16, device=W.device)
    lib = load()
    with torch.cuda.device(W.device):
        check("q8_0_quantize", lib.q8_0_quantize(_ptr(W), N, K, _ptr(qs), _ptr(d),
                                                 _stream(W.device)))
    return qs, d


def q8_0_dequantize(qs: torch.Tensor, d: torch.Tensor,
                    out: torch.Tensor | None = None) -> torch.Tensor:
    """bf16(d * q) as bf16 [N, K]."""
    _need(qs, "qs", torch.int8, 2)
    N, K = qs.shape
    _need(d, "d", torch.float16, 2, qs.device)
    if tuple(d.shape) != (N, K // Q8_0_BLOCK):
        raise ValueError("d must be [N, K/32]")
    W = _out(out, (N, K), torch.bfloat16, qs.device, "out")
    lib = load()
    with torch.cuda.device(qs.device):
        check("q8_0_dequantize", lib.q8_0_dequantize(_ptr(qs), _ptr(d), N, K, _ptr(W),
                                                     _stream(qs.device)))
    return W


def q8_0_linear(X: torch.Tensor, qs: torch.Tensor, d: torch.Tensor,
                bias: torch.Tensor | None = None, work: torch.Tensor | None = None,
                out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X W'^T + bias with W' = bf16(d * q) decoded into `work` (bf16
    [N, K], allocated if not given)."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    _need(qs, "qs", torch.int8, 2, X.device)
    N = qs.shape[0]
    if qs.shape[1] != K:
        raise ValueError("qs must be [N, K]")
    _need(d, "d", torch.float16, 2, X.device)
    if tuple(d.shape) != (N, K // Q8_0_BLOCK):
        raise ValueError("d must be [N, K/32]")
    if bias is not None:
        _need_vec(bias, "bias", torch.bfloat16, N, X.device)
    work = _out(work, (N, K), torch.bfloat16, X.device, "work")
    Y = _out(out, (M, N), torch.bfloat16, X.device, "out")
    lib = load()
    with torch.cuda.device(X.device):
        check("q8_0_linear", lib.q8_0_linear(_ptr(X), _ptr(qs), _ptr(d), _ptr(bias), M, N, K,
                                             _ptr(work), _ptr(Y), _stream(X.device)))
    return Y


# --------------------------------------------------------------------------
# GGUF Q4_K weight-only
# --------------------------------------------------------------------------

Q4_K_SUPER = 256
Q4_K_SUB = 32


class Q4K:
    """The planes of a Q4_K weight [N, K]: qs uint8 [N, K/2] (two 4-bit codes
    per byte, even k low), scales uint8 [N, K/256 * 12] (each super-block's
    eight 6-bit sub-block scales and offsets, packed), d and dmin float16
    [N, K/256] (super-block scales): 4.5 bits per weight."""

    __slots__ = ("qs", "scales", "d", "dmin")

    def __init__(self, qs, scales, d, dmin):
        self.qs, self.scales, self.d, self.dmin = qs, scales, d, dmin

    @property
    def shape(self) -> tuple[int, int]:
        return self.qs.shape[0], 2 * self.qs.shape[1]

    @property
    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in (self.qs, self.scales, self.d, self.dmin))

    def check(self, device=None) -> tuple[int, int]:
        _need(self.qs, "qs", torch.uint8, 2, device)
        N, K = self.shape
        dev = self.qs.device
        for name, t, dt, cols in (("scales", self.scales, torch.uint8, K // Q4_K_SUPER * 12),
                                  ("d", self.d, torch.float16, K // Q4_K_SUPER),
                                  ("dmin", self.dmin, torch.float16, K // Q4_K_SUPER)):
            _need(t, name, dt, 2, dev)
            if tuple(t.shape) != (N, cols):
                raise ValueError(f"{name} must be [{N}, {cols}], got {tuple(t.shape)}")
        return N, K

    def ptrs(self):
        return [_ptr(t) for t in (self.qs, self.scales, self.d, self.dmin)]


def q4_k_quantize(W: torch.Tensor) -> Q4K:
    """W [N, K] bf16 (256 | K) -> its Q4_K planes."""
    _need(W, "W", torch.bfloat16, 2)
    N, K = W.shape
    dev = W.device
    q = Q4K(torch.empty(N, K // 2, dtype=torch.uint8, device=dev),
            torch.empty(N, K // Q4_K_SUPER * 12, dtype=torch.uint8, device=dev),
            torch.empty(N, K // Q4_K_SUPER, dtype=torch.float16, device=dev),
            torch.empty(N, K // Q4_K_SUPER, dtype=torch.float16, device=dev))
    lib = load()
    with torch.cuda.device(dev):
        check("q4_k_quantize", lib.q4_k_quantize(_ptr(W), N, K, *q.ptrs(), _stream(dev)))
    return q


def q4_k_dequantize(q: Q4K, out: torch.Tensor | None = None) -> torch.Tensor:
    """bf16(d * sc * code - dmin * m) as bf16 [N, K]."""
    N, K = q.check()
    dev = q.qs.device
    W = _out(out, (N, K), torch.bfloat16, dev, "out")
    lib = load()
    with torch.cuda.device(dev):
        check("q4_k_dequantize", lib.q4_k_dequantize(*q.ptrs(), N, K, _ptr(W), _stream(dev)))
    return W


def q4_k_linear(X: torch.Tensor, q: Q4K, bias: torch.Tensor | None = None,
                work: torch.Tensor | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = X W'^T + bias with W' the decoded Q4_K weights, decoded into
    `work` (bf16 [N, K], allocated if not given)."""
    _need(X, "X", torch.bfloat16, 2)
    M, K = X.shape
    N, Kq = q.check(X.device)
    if Kq != K:
        raise ValueError(f"the weights are [{N}, {Kq}], X has K = {K}")
    if bias is not None:
        _need_vec(bias, "bias", torch.bfloat16, N, X.device)
    work = _out(work, (N, K), torch.bfloat16, X.device, "work")
    Y = _out(out, (M, N), torch.bfloat16, X.device, "out")
    lib = load()
    with torch.cuda.device(X.device):
        check("q4_k_linear", lib.q4_k_linear(_ptr(X), *q.ptrs(), _ptr(bias), M, N, K,
                                             _ptr(work), _ptr(Y), _stream(X.device)))
    return Y
