"""Activation-fragility profiling and protection (paper Section 3).

Every linear's input is profiled per denoising step: its max |x|, standard
deviation and kurtosis, computed on the GPU by w8a8_act_moments. A layer's
fragility score is its kurtosis averaged over the profiled steps; the N
highest-scoring layers are kept in bf16 (no activation quantization), the
rest run W8A8. The ranking's stability over the trajectory is checked with
the Spearman rank correlation of scores from early and late steps.

Selection and ranking are host logic over a few hundred numbers.
"""
from __future__ import annotations

import numpy as np
import torch

from . import ops
from ._lib import MOMENTS_WORK_BYTES

MAX_ABS, MEAN, STD, KURTOSIS = range(4)


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
        """Fragility score per layer over the given steps."""
        return fragility_scores(self.table()[:, steps, KURTOSIS])


def fragility_scores(kurtosis) -> np.ndarray:
    """Mean kurtosis over steps; kurtosis is [layers, steps]."""
    k = np.asarray(kurtosis, dtype=np.float64)
    return k.mean(axis=1)


def select_protected(scores, n: int) -> list[int]:
    """The n most fragile layers, most fragile first (equal scores: lower
    layer index first)."""
    s = np.asarray(scores, dtype=np.float64)
    order = np.lexsort((np.arange(s.size), -s))
    return [int(i) for i in order[: max(0, n)]]


def _average_ranks(v: np.ndarray) -> np.ndarray:
    order = np.argsort(v, kind="stable")
    ranks = np.empty(v.size, dtype=np.float64)
    sv = v[order]
    start = 0
    for end in range(1, v.size + 1):
        if end == v.size or sv[end] != sv[start]:
            ranks[order[start:end]] = 0.5 * (start + end - 1) + 1.0
            start = end
    return ranks


def rank_stability(scores_a, scores_b) -> float:
    """Spearman rank correlation between two score vectors (average ranks
    for ties)."""
    ra = _average_ranks(np.asarray(scores_a, dtype=np.float64))
    rb = _average_ranks(np.asarray(scores_b, dtype=np.float64))
    ra -= ra.mean()
    rb -= rb.mean()
    return float((ra * rb).sum() / np.sqrt((ra * ra).sum() * (rb * rb).sum()))
