"""Activation-fragility profiling and protection (paper Section 3).

Every linear's input is profiled per denoising step: its max |x|, standard
deviation and kurtosis, computed on the GPU by w8a8_act_moments. A layer's
fragility score is its kurtosis averaged over the profiled steps; the N
highest-scoring layers are kept in bf16 (no activation quantization), the
rest run W8A8. The ranking's stability over the trajectory is checked with
the Spearman rank correlation of scores from early and late steps.

Argument marshalling only: the scores, the selection and the rank
correlation are the library's host calls w8a8_fragility_scores,
w8a8_select_protected and w8a8_rank_correlation (include/w8a8.h).
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import ops
from ._lib import MOMENTS_WORK_BYTES, check, load

MAX_ABS, MEAN, STD, KURTOSIS = range(4)


def _host_f64(a, name: str, ndim: int) -> np.ndarray:
    v = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    if v.ndim != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got shape {v.shape}")
    return v


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class Profile:
    """Per (layer, step) statistics, kept on the device until read."""

    def __init__(self, n_layers: int, n_steps: int, device):
        self.stats = torch.zeros(n_layers, n_steps, 4, dtype=torch.float64, device=device)
        self.work = torch.empty(MOMENTS_WORK_BYTES, dtype=torch.uint8, device=device)

    def record(self, layer: int, step: int, X: torch.Tensor) -> None:
        """Statistics of the input X [tokens, features] of `layer` at `step`
        (asynchronous on the current stream)."""
        ops.w8a8_act_moments(X, self.work, out=self.stats[layer, step])

    def table(self) -> np.ndarray:
        """[layers, steps, 4]: max |x|, mean, std, kurtosis."""
        return self.stats.cpu().numpy()

    def scores(self, steps: slice = slice(None)) -> np.ndarray:
        """Fragility score per layer over a contiguous range of steps."""
        n_steps = self.stats.shape[1]
        begin, end, stride = steps.indices(n_steps)
        if stride != 1:
            raise ValueError("steps must be a contiguous range")
        return fragility_scores(self.table()[:, :, KURTOSIS], begin, end)


def fragility_scores(kurtosis, step_begin: int = 0, step_end: int | None = None) -> np.ndarray:
    """Mean kurtosis over steps [step_begin, step_end) of kurtosis [layers, steps]."""
    k = _host_f64(kurtosis, "kurtosis", 2)
    layers, steps = k.shape
    end = steps if step_end is None else step_end
    out = np.empty(layers, dtype=np.float64)
    check("w8a8_fragility_scores",
          load().w8a8_fragility_scores(_dp(k), layers, steps, step_begin, end, _dp(out)))
    return out


def select_protected(scores, n: int) -> list[int]:
    """The n most fragile layers, most fragile first (equal scores: lower
    layer index first); all of them when n exceeds the layer count."""
    s = _host_f64(scores, "scores", 1)
    n = max(0, min(int(n), s.size))
    idx = np.empty(max(n, 1), dtype=np.int32)
    check("w8a8_select_protected", load().w8a8_select_protected(_dp(s), s.size, n, _dp(idx)))
    return [int(i) for i in idx[:n]]


def rank_stability(scores_a, scores_b) -> float:
    """Spearman rank correlation between two score vectors (average ranks
    for ties)."""
    a = _host_f64(scores_a, "scores_a", 1)
    b = _host_f64(scores_b, "scores_b", 1)
    if a.size != b.size:
        raise ValueError("the two score vectors must have the same length")
    rho = ctypes.c_double()
    check("w8a8_rank_correlation",
          load().w8a8_rank_correlation(_dp(a), _dp(b), a.size, ctypes.byref(rho)))
    return rho.value
