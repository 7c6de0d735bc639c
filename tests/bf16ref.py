"""Exact bf16 rounding by brute force, for pinning the oracle's conversions.

Every finite bf16 value is enumerated; a binary64 input is rounded to the
nearest one by exact rational comparison (ties to the even bit pattern). This
is independent of both the oracle and the GPU library."""
from __future__ import annotations

from fractions import Fraction

import numpy as np

_POS_BITS = np.arange(0x0000, 0x7F80, dtype=np.uint32)       # +0 .. max finite
_POS_VALS = (_POS_BITS << 16).view(np.float32).astype(np.float64)
_MAX = Fraction(float(_POS_VALS[-1]))
_OVERFLOW = _MAX + (Fraction(2) ** 128 - _MAX) / 2            # midpoint to 2^128


def round_bf16_exact(d) -> int:
    """Nearest bf16 bit pattern of a finite number (float or Fraction)."""
    x = Fraction(d)
    if x == 0:
        if isinstance(d, float) and np.signbit(d):
            return 0x8000
        return 0x0000
    sign = 0x8000 if x < 0 else 0
    a = abs(x)
    if a >= _OVERFLOW:
        return sign | 0x7F80
    i = int(np.searchsorted(_POS_VALS, float(a)))
    cands = [j for j in (i - 1, i, i + 1) if 0 <= j < len(_POS_VALS)]
    best = None
    for j in cands:
        dist = abs(Fraction(float(_POS_VALS[j])) - a)
        key = (dist, int(_POS_BITS[j]) & 1)
        if best is None or key < best[0]:
            best = (key, j)
    return sign | int(_POS_BITS[best[1]])


def bf16_to_f64(h) -> np.ndarray:
    return (np.asarray(h, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def ulp_distance(a, b) -> np.ndarray:
    """Distance in bf16 ulps between two bf16 bit-pattern arrays (ordered
    integer mapping, so -0 and +0 are 0 apart)."""
    def key(h):
        h = np.asarray(h, np.uint16).astype(np.int64)
        neg = (h & 0x8000) != 0
        mag = h & 0x7FFF
        return np.where(neg, -mag, mag)
    return np.abs(key(a) - key(b))
