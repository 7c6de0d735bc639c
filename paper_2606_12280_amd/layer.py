"""One linear of the DiT routed through the W8A8 recipe or the protected bf16
path (paper Section 3: every linear is W8A8 except the top-N most fragile
layers, N = 17 of 211 per branch, which stay bf16 with no activation
quantization). Host-side bookkeeping only: the arithmetic runs in the
library's kernels through ops."""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import ops


@dataclass
class PreparedLinear:
    """The per-layer bundle kept resident in HBM."""
    protected: bool
    N: int
    K: int
    bias: torch.Tensor | None
    W: torch.Tensor | None = None            # bf16 [N, K], protected layers only
    Wq: torch.Tensor | None = None           # int8 [N, K]
    w_scale: torch.Tensor | None = None      # fp32 [N]
    inv_lambda: torch.Tensor | None = None   # fp32 [K]

    def nbytes(self) -> int:
        ts = [self.W, self.Wq, self.w_scale, self.inv_lambda, self.bias]
        return sum(t.numel() * t.element_size() for t in ts if t is not None)


def prepare_linear(W: torch.Tensor, bias: torch.Tensor | None, lam: torch.Tensor | None,
                   protected: bool) -> PreparedLinear:
    """Quantize W once (offline) unless the layer is protected. ``lam`` is the
    smoothing vector (None: no smoothing, lambda = 1)."""
    N, K = W.shape
    if protected:
        return PreparedLinear(True, N, K, bias, W=W)
    if lam is None:
        lam = torch.ones(K, dtype=torch.float32, device=W.device)
    Wq, ws, il = ops.w8a8_prepare_weight(W, lam)
    return PreparedLinear(False, N, K, bias, Wq=Wq, w_scale=ws, inv_lambda=il)


class Workspace:
    """Reusable activation buffers (Xq, x_scale) so that a forward allocates
    nothing once the largest shape has been seen."""

    def __init__(self, device):
        self.device = device
        self._xq = None
        self._xs = None

    def get(self, M: int, K: int):
        need = M * K
        if self._xq is None or self._xq.numel() < need:
            self._xq = torch.empty(need, dtype=torch.int8, device=self.device)
        if self._xs is None or self._xs.numel() < M:
            self._xs = torch.empty(M, dtype=torch.float32, device=self.device)
        return self._xq[:need].view(M, K), self._xs[:M]


def route(layer: PreparedLinear, X: torch.Tensor, out: torch.Tensor | None = None,
          ws: Workspace | None = None) -> torch.Tensor:
    """Y = layer(X): bf16_linear for a protected layer, else quant + W8A8 GEMM."""
    if layer.protected:
        return ops.bf16_linear(X, layer.W, layer.bias, out=out)
    M = X.shape[0]
    if ws is None:
        Xq = x_scale = None
    else:
        Xq, x_scale = ws.get(M, layer.K)
    Xq, x_scale = ops.w8a8_quant_act(X, layer.inv_lambda, Xq=Xq, x_scale=x_scale)
    return ops.w8a8_linear(Xq, x_scale, layer.Wq, layer.w_scale, layer.bias, out=out)


def protected_layers(n_layers: int, n_protect: int, shapes_cycle: int = 4,
                     down_slot: int = 3) -> list[bool]:
    """Protection flags for a backbone whose layers cycle over
    ``shapes_cycle`` block shapes: the first ``n_protect`` FFN
    down-projections (slot ``down_slot``) in layer order are protected."""
    flags = [False] * n_layers
    left = n_protect
    for i in range(n_layers):
        if left and i % shapes_cycle == down_slot:
            flags[i] = True
            left -= 1
    return flags
