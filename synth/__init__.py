"""Seeded synthetic inputs for the W8A8 linear workloads.

This module only draws random tensors: it holds none of the quantization
arithmetic. The same host arrays feed the CPU oracle and the GPU library.
Random values are drawn in float32 with NumPy's PCG64 generator and rounded
to bf16 by torch's round-to-nearest-even conversion. bf16 tensors are returned
as ``uint16`` arrays of bit patterns.

The shapes and distributions stand in for the activations and weights of the
paper's dual-branch DiT (Section 3, "Setting": 211 linears per branch, two
separate-weight branches), whose checkpoints are not available: tokens
M = 4608 (4096 image + 512 text), widths 4096 / 12288 / 16384.
"""
from __future__ import annotations

import numpy as np
import torch

TOKENS = 4608

# (name, N_out, K_in) of the four linears of one DiT block, in layer order.
BLOCK_SHAPES = (
    ("qkv", 12288, 4096),
    ("attn_out", 4096, 4096),
    ("ffn_up", 16384, 4096),
    ("ffn_down", 4096, 16384),
)


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 array -> bf16 bit patterns (uint16), round to nearest even."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact widening)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def outlier_activations(rng, M: int, K: int, n_outlier: int, factor: float) -> np.ndarray:
    """N(0,1) tokens with ``n_outlier`` channels scaled by ``factor``.

    The channel indices are drawn right after X."""
    x = normal(rng, (M, K), 1.0)
    if n_outlier > 0:
        idx = rng.choice(K, n_outlier, replace=False)
        x[:, idx] *= np.float32(factor)
    return x


def gelu_lognormal_activations(rng, M: int, K: int, sigma_z=1.5, sigma_c=1.5) -> np.ndarray:
    """Post-GELU-like activations with heavy-tailed per-channel scales:
    GELU(z) * c_j, z ~ N(0, sigma_z), c_j ~ LogNormal(0, sigma_c)."""
    z = torch.from_numpy(normal(rng, (M, K), sigma_z))
    g = torch.nn.functional.gelu(z).numpy()
    c = rng.lognormal(0.0, sigma_c, size=K).astype(np.float32)
    g *= c[None, :]
    return g


def linear_case(seed, M: int, N: int, K: int, act: str = "outlier",
                n_outlier: int | None = None, outlier_factor: float = 20.0,
                w_std: float = 0.02, b_std: float = 0.01, bias: bool = True) -> dict:
    """One linear: X [M][K], W [N][K], bias [N] as bf16 bits.

    act = "outlier": N(0,1) with round(1% of K) channels x outlier_factor
          (or ``n_outlier`` channels); "gelu": GELU(N(0,1.5)) * LogNormal(0,1.5)
          per channel; "normal": plain N(0,1)."""
    rng = np.random.default_rng(seed)
    if act == "outlier":
        n_out = int(round(0.01 * K)) if n_outlier is None else n_outlier
        x = outlier_activations(rng, M, K, n_out, outlier_factor)
    elif act == "gelu":
        x = gelu_lognormal_activations(rng, M, K)
    elif act == "normal":
        x = normal(rng, (M, K), 1.0)
    else:
        raise ValueError(act)
    w = normal(rng, (N, K), w_std)
    case = {"X": to_bf16_bits(x), "W": to_bf16_bits(w), "M": M, "N": N, "K": K}
    case["bias"] = to_bf16_bits(normal(rng, (N,), b_std)) if bias else None
    return case


def tiny_case() -> dict:
    """Tiny linear: X [64 x 256] N(0,1) with 4 outlier channels x30,
    W [512 x 256] N(0,0.02), bias N(0,0.01); seed 0; draw order X, idx, W, bias."""
    return linear_case(0, 64, 512, 256, act="outlier", n_outlier=4, outlier_factor=30.0)


def ffn_up_case(M: int = TOKENS) -> dict:
    """DiT FFN up-projection, one branch: X [4608 x 4096] N(0,1) with 1% of the
    channels x20, W [16384 x 4096] N(0,0.02), bias N(0,0.01)."""
    return linear_case([2], M, 16384, 4096, act="outlier", outlier_factor=20.0)


def ffn_down_case(M: int = TOKENS) -> dict:
    """Fragile FFN down-projection: X [4608 x 16384] GELU(N(0,1.5)) times
    LogNormal(0,1.5) channel scales, W [4096 x 16384] N(0,0.02)."""
    return linear_case([3], M, 4096, 16384, act="gelu")


def block_case(branch: int, layer: int, M: int = TOKENS) -> dict:
    """Linear ``layer`` (0..3: qkv, attn_out, ffn_up, ffn_down) of one DiT
    block for CFG branch ``branch`` (0 cond, 1 uncond), independent seeds."""
    name, N, K = BLOCK_SHAPES[layer]
    act = "gelu" if name == "ffn_down" else "outlier"
    c = linear_case([4, branch, layer], M, N, K, act=act)
    c["name"] = name
    return c


def rand_bf16(seed, shape, std: float = 1.0) -> np.ndarray:
    """Plain N(0, std) bf16 bits of any shape (edge-case tests)."""
    rng = np.random.default_rng(seed)
    return to_bf16_bits(normal(rng, shape, std))


def rand_i8(seed, shape) -> np.ndarray:
    """Uniform int8 codes in [-127, 127] (GEMM-only tests)."""
    rng = np.random.default_rng(seed)
    return rng.integers(-127, 128, size=shape, dtype=np.int8)
