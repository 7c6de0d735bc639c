"""CPU oracle of the INT8 W8A8 linear -- TEST INFRASTRUCTURE.

Only tests/, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. It wraps ``liboracle.so`` (built from
``oracle.c`` by :func:`build`) with NumPy-array functions. It shares no code
with the GPU library.

bf16 tensors are ``uint16`` arrays of bit patterns. Every function returns new
arrays and follows the step of the paper's Section 3 recipe named in its
docstring (see ``oracle.c`` for the arithmetic and the readings it takes).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
          "-shared", "-fPIC", "-std=c11", "-Wall", "-Wextra"]


def build() -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    tmp = f"{_LIB_PATH}.{os.getpid()}.tmp"   # parallel test workers each build their own
    subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def use_library(path: str | None) -> None:
    """Point the wrappers at another build of oracle.c (None: the default).
    Used only by the mutation test, which plants mistakes in copies."""
    global _lib, _lib_override
    _lib_override = path
    _lib = None


_lib_override = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = _lib_override or _LIB_PATH
    if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    sig = {
        "oracle_num_threads": ([], ctypes.c_int),
        "oracle_set_num_threads": ([ctypes.c_int], None),
        "oracle_bf16_to_float": ([ctypes.c_uint16], ctypes.c_float),
        "oracle_double_to_bf16": ([ctypes.c_double], ctypes.c_uint16),
        "oracle_act_absmax": ([P, I64, I64, P], None),
        "oracle_smooth_factors": ([P, P, I64, I64, ctypes.c_double, P], None),
        "oracle_prepare_weight": ([P, P, I64, I64, P, P, P], None),
        "oracle_quant_act": ([P, P, I64, I64, P, P], None),
        "oracle_gemm_i32": ([P, P, I64, I64, I64, P], None),
        "oracle_epilogue": ([P, P, P, P, I64, I64, P], None),
        "oracle_w8a8_linear": ([P, P, P, P, P, I64, I64, I64, P], None),
        "oracle_bf16_linear": ([P, P, P, I64, I64, I64, P], None),
        "oracle_act_moments": ([P, I64, I64, P], ctypes.c_int),
        "oracle_float_to_half": ([ctypes.c_float], ctypes.c_uint16),
        "oracle_half_to_float": ([ctypes.c_uint16], ctypes.c_float),
        "oracle_q8_0_quantize": ([P, I64, I64, P, P], None),
        "oracle_q8_0_dequantize": ([P, P, I64, I64, P], None),
        "oracle_adaln_modulate": ([P, P, P, I64, I64, ctypes.c_double, P], None),
        "oracle_q4_k_quantize": ([P, I64, I64, P, P, P, P], None),
        "oracle_q4_k_dequantize": ([P, P, P, P, I64, I64, P], None),
        "oracle_q4_k_pack_scales": ([P, P, P], None),
        "oracle_q4_k_unpack_scales": ([P, P, P], None),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return _load().oracle_num_threads()


def set_num_threads(n: int) -> None:
    _load().oracle_set_num_threads(int(n))


def bf16_to_float(h: int) -> float:
    return float(_load().oracle_bf16_to_float(int(h)))


def double_to_bf16(d: float) -> int:
    return int(_load().oracle_double_to_bf16(float(d)))


def act_absmax(X, M: int, K: int, s=None) -> np.ndarray:
    """Calibration statistic s_j = max_t |X_tj| (Section 3, "INT8 W8A8": the
    activation scales are measured beforehand on calibration inputs),
    accumulated into ``s`` if given."""
    X = _c(X, np.uint16)
    out = np.zeros(K, np.float32) if s is None else np.array(s, np.float32, copy=True)
    _load().oracle_act_absmax(_p(X), M, K, _p(out))
    return out


def smooth_factors(act_absmax_, W, N: int, K: int, alpha: float = 0.5) -> np.ndarray:
    """lambda_j = s_j^alpha / max_i |W_ij|^(1-alpha) (Section 3, the
    smoothing equation), binary64 rounded once to binary32."""
    s = _c(act_absmax_, np.float32)
    W = _c(W, np.uint16)
    lam = np.empty(K, np.float32)
    _load().oracle_smooth_factors(_p(s), _p(W), N, K, float(alpha), _p(lam))
    return lam


def prepare_weight(W, lam, N: int, K: int):
    """Offline weight side (Section 3): W*diag(lambda), per-output-row
    symmetric INT8 with round to nearest. Returns (Wq, w_scale, inv_lambda)."""
    W = _c(W, np.uint16)
    lam = _c(lam, np.float32)
    Wq = np.empty((N, K), np.int8)
    ws = np.empty(N, np.float32)
    il = np.empty(K, np.float32)
    _load().oracle_prepare_weight(_p(W), _p(lam), N, K, _p(Wq), _p(ws), _p(il))
    return Wq, ws, il


def quant_act(X, inv_lam, M: int, K: int):
    """Runtime activation side (Section 3): X*diag(1/lambda), per-token
    dynamic symmetric INT8. Returns (Xq, x_scale)."""
    X = _c(X, np.uint16)
    il = _c(inv_lam, np.float32)
    Xq = np.empty((M, K), np.int8)
    xs = np.empty(M, np.float32)
    _load().oracle_quant_act(_p(X), _p(il), M, K, _p(Xq), _p(xs))
    return Xq, xs


def adaln_modulate(X, shift, scale, M: int, K: int, eps: float = 1e-6) -> np.ndarray:
    """bf16 bits [M][K] of LayerNorm(X) * (1 + scale) + shift (binary64, one
    rounding to bf16)."""
    X = _c(X, np.uint16)
    H = np.empty((M, K), np.uint16)
    _load().oracle_adaln_modulate(_p(X), _p(_c(shift, np.uint16)), _p(_c(scale, np.uint16)),
                                  M, K, float(eps), _p(H))
    return H


def adaln_quant_act(X, shift, scale, inv_lam, M: int, K: int, eps: float = 1e-6):
    """The W8A8 activation side on the adaLN-modulated input: quant_act of
    adaln_modulate(X). Returns (Xq, x_scale)."""
    return quant_act(adaln_modulate(X, shift, scale, M, K, eps), inv_lam, M, K)


def gemm_i32(Xq, Wq, M: int, N: int, K: int) -> np.ndarray:
    """acc = Xq Wq^T with exact int32 accumulation."""
    Xq = _c(Xq, np.int8)
    Wq = _c(Wq, np.int8)
    C = np.empty((M, N), np.int32)
    _load().oracle_gemm_i32(_p(Xq), _p(Wq), M, N, K, _p(C))
    return C


def epilogue(C, x_scale, w_scale, bias, M: int, N: int) -> np.ndarray:
    """y = bf16(acc * s_tok * s_ch + bias), one rounding from binary64."""
    C = _c(C, np.int32)
    xs = _c(x_scale, np.float32)
    ws = _c(w_scale, np.float32)
    b = None if bias is None else _c(bias, np.uint16)
    Y = np.empty((M, N), np.uint16)
    _load().oracle_epilogue(_p(C), _p(xs), _p(ws), _p(b), M, N, _p(Y))
    return Y


def w8a8_linear(Xq, x_scale, Wq, w_scale, bias, M: int, N: int, K: int) -> np.ndarray:
    """The int32 product and the epilogue, fused per row."""
    Xq = _c(Xq, np.int8)
    Wq = _c(Wq, np.int8)
    xs = _c(x_scale, np.float32)
    ws = _c(w_scale, np.float32)
    b = None if bias is None else _c(bias, np.uint16)
    Y = np.empty((M, N), np.uint16)
    _load().oracle_w8a8_linear(_p(Xq), _p(xs), _p(Wq), _p(ws), _p(b), M, N, K, _p(Y))
    return Y


def bf16_linear(X, W, bias, M: int, N: int, K: int) -> np.ndarray:
    """Protected layer (Section 3): bf16(X W^T + bias), binary64 sum."""
    X = _c(X, np.uint16)
    W = _c(W, np.uint16)
    b = None if bias is None else _c(bias, np.uint16)
    Y = np.empty((M, N), np.uint16)
    _load().oracle_bf16_linear(_p(X), _p(W), _p(b), M, N, K, _p(Y))
    return Y


def recipe(X, W, bias, M: int, N: int, K: int, alpha: float = 0.5, lam=None):
    """The whole W8A8 recipe on one linear, calibrated on X itself:
    returns a dict of every intermediate (lambda, inv_lambda, Wq, w_scale,
    Xq, x_scale, acc, Y)."""
    if lam is None:
        lam = smooth_factors(act_absmax(X, M, K), W, N, K, alpha)
    Wq, ws, il = prepare_weight(W, lam, N, K)
    Xq, xs = quant_act(X, il, M, K)
    acc = gemm_i32(Xq, Wq, M, N, K)
    Y = epilogue(acc, xs, ws, bias, M, N)
    return {"lambda": lam, "inv_lambda": il, "Wq": Wq, "w_scale": ws,
            "Xq": Xq, "x_scale": xs, "acc": acc, "Y": Y}


# --------------------------------------------------------------------------
# fragility profile and protection (Section 3, "Activation-fragility
# profiling and protection")
# --------------------------------------------------------------------------

def act_moments(X, M: int, K: int) -> np.ndarray:
    """[max |x|, mean, population std, Pearson kurtosis] of the M*K bf16
    entries of X, binary64, two passes (kurtosis 0 for a constant input)."""
    X = _c(X, np.uint16)
    out = np.zeros(4, np.float64)
    rc = _load().oracle_act_moments(_p(X), M, K, _p(out))
    if rc != 0:
        raise MemoryError("oracle_act_moments")
    return out


def fragility_scores(kurtosis) -> np.ndarray:
    """A layer's fragility score: its activation kurtosis averaged over the
    profiled denoising steps. kurtosis is [layers][steps]."""
    k = np.asarray(kurtosis, np.float64)
    return k.sum(axis=1) / k.shape[1]


def top_n(scores, n: int) -> list[int]:
    """Indices of the n most fragile layers: largest score first, equal
    scores by lower layer index."""
    s = [float(v) for v in scores]
    order = sorted(range(len(s)), key=lambda i: (-s[i], i))
    return order[:n]


def _ranks(v) -> list[float]:
    """1-based ranks, equal values sharing the mean of their positions."""
    v = [float(x) for x in v]
    order = sorted(range(len(v)), key=lambda i: v[i])
    r = [0.0] * len(v)
    i = 0
    while i < len(order):
        j = i
        while j + 1 < len(order) and v[order[j + 1]] == v[order[i]]:
            j += 1
        for q in range(i, j + 1):
            r[order[q]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return r


def spearman(a, b) -> float:
    """Spearman rank correlation: the Pearson correlation of the ranks (the
    paper's check that the ranking is stable between early and late steps)."""
    ra, rb = _ranks(a), _ranks(b)
    n = len(ra)
    ma, mb = sum(ra) / n, sum(rb) / n
    cov = sum((x - ma) * (y - mb) for x, y in zip(ra, rb))
    va = sum((x - ma) ** 2 for x in ra)
    vb = sum((y - mb) ** 2 for y in rb)
    return cov / (va * vb) ** 0.5


# --------------------------------------------------------------------------
# GGUF Q8_0 weight-only (Section 3, "GGUF k-quants")
# --------------------------------------------------------------------------

Q8_0_BLOCK = 32


def float_to_half(f: float) -> int:
    return int(_load().oracle_float_to_half(float(f)))


def half_to_float(h: int) -> float:
    return float(_load().oracle_half_to_float(int(h)))


def q8_0_quantize(W, N: int, K: int):
    """W [N][K] bf16 bits -> (codes int8 [N][K], scales binary16 bits [N][K/32])."""
    W = _c(W, np.uint16)
    qs = np.zeros(N * K, np.int8)
    d = np.zeros(N * (K // Q8_0_BLOCK), np.uint16)
    _load().oracle_q8_0_quantize(_p(W), N, K, _p(qs), _p(d))
    return qs.reshape(N, K), d.reshape(N, K // Q8_0_BLOCK)


def q8_0_dequantize(qs, d, N: int, K: int) -> np.ndarray:
    """bf16 bits [N][K] of bf16(d * q)."""
    qs = _c(qs, np.int8)
    d = _c(d, np.uint16)
    W = np.zeros(N * K, np.uint16)
    _load().oracle_q8_0_dequantize(_p(qs), _p(d), N, K, _p(W))
    return W.reshape(N, K)


def q8_0_linear(X, qs, d, bias, M: int, N: int, K: int) -> np.ndarray:
    """The weight-only linear: bf16 X times the dequantized weights (the
    protected-layer arithmetic on bf16(d * q))."""
    return bf16_linear(X, q8_0_dequantize(qs, d, N, K), bias, M, N, K)


Q4_K_SUPER = 256
Q4_K_SUB = 32


def q4_k_quantize(W, N: int, K: int):
    """W [N][K] bf16 bits -> dict of the Q4_K planes: qs uint8 [N][K/2] (two
    4-bit codes per byte, even k low), scales uint8 [N][K/256 * 12] (each
    super-block's eight 6-bit sub-block scales and offsets, packed), d and
    dmin binary16 bits [N][K/256]."""
    W = _c(W, np.uint16)
    qs = np.zeros(N * K // 2, np.uint8)
    scales = np.zeros(N * (K // Q4_K_SUPER) * 12, np.uint8)
    d = np.zeros(N * (K // Q4_K_SUPER), np.uint16)
    dmin = np.zeros(N * (K // Q4_K_SUPER), np.uint16)
    _load().oracle_q4_k_quantize(_p(W), N, K, _p(qs), _p(scales), _p(d), _p(dmin))
    return {"qs": qs.reshape(N, K // 2), "scales": scales.reshape(N, (K // Q4_K_SUPER) * 12),
            "d": d.reshape(N, K // Q4_K_SUPER), "dmin": dmin.reshape(N, K // Q4_K_SUPER)}


def q4_k_pack_scales(sc, mn) -> np.ndarray:
    """The 12 bytes holding eight 6-bit sub-block scales and offsets."""
    sc = _c(np.asarray(sc).reshape(8), np.uint8)
    mn = _c(np.asarray(mn).reshape(8), np.uint8)
    out = np.zeros(12, np.uint8)
    _load().oracle_q4_k_pack_scales(_p(sc), _p(mn), _p(out))
    return out


def q4_k_unpack_scales(packed):
    """(sc [8], mn [8]) from 12 packed bytes."""
    packed = _c(np.asarray(packed).reshape(12), np.uint8)
    sc = np.zeros(8, np.uint8)
    mn = np.zeros(8, np.uint8)
    _load().oracle_q4_k_unpack_scales(_p(packed), _p(sc), _p(mn))
    return sc, mn


def q4_k_sub_scales(q, N: int, K: int):
    """The planes' sub-block scales and offsets unpacked: (sc, mn), each
    uint8 [N][K/32]."""
    sb = K // Q4_K_SUPER
    packed = np.asarray(q["scales"], np.uint8).reshape(N * sb, 12)
    sc = np.zeros((N * sb, 8), np.uint8)
    mn = np.zeros((N * sb, 8), np.uint8)
    for i in range(N * sb):
        sc[i], mn[i] = q4_k_unpack_scales(packed[i])
    return sc.reshape(N, K // Q4_K_SUB), mn.reshape(N, K // Q4_K_SUB)


def q4_k_dequantize(q, N: int, K: int) -> np.ndarray:
    """bf16 bits [N][K] of bf16(RN32(d * sc * code - dmin * mn))."""
    planes = [_c(q["qs"], np.uint8), _c(q["scales"], np.uint8), _c(q["d"], np.uint16),
              _c(q["dmin"], np.uint16)]
    W = np.zeros(N * K, np.uint16)
    _load().oracle_q4_k_dequantize(*[_p(a) for a in planes], N, K, _p(W))
    return W.reshape(N, K)


def q4_k_linear(X, q, bias, M: int, N: int, K: int) -> np.ndarray:
    """The weight-only linear on the decoded Q4_K weights."""
    return bf16_linear(X, q4_k_dequantize(q, N, K), bias, M, N, K)
