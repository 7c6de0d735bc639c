"""One linear of the DiT routed through the W8A8 recipe, the protected bf16
path, or a GGUF weight-only format, Q8_0 or Q4_K (paper Section 3: every
linear is W8A8 except the top-N most fragile layers, N = 17 of 211 per
branch, which stay bf16 with no activation quantization; independently, a
checkpoint can be stored as Q8_0 or Q4_K). Host-side bookkeeping only: the
arithmetic runs in the library's kernels through ops."""
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
    q8_qs: torch.Tensor | None = None        # int8 [N, K], Q8_0 layers only
    q8_d: torch.Tensor | None = None         # fp16 [N, K/32]
    q4k: ops.Q4K | None = None               # Q4_K planes, Q4_K layers only

    @property
    def q8_0(self) -> bool:
        return self.q8_qs is not None

    @property
    def weight_only(self) -> bool:
        """A GGUF layer: decoded to bf16, then the bf16 linear."""
        return self.q8_qs is not None or self.q4k is not None

    def nbytes(self) -> int:
        ts = [self.W, self.Wq, self.w_scale, self.inv_lambda, self.bias, self.q8_qs, self.q8_d]
        n = sum(t.numel() * t.element_size() for t in ts if t is not None)
        return n + (self.q4k.nbytes if self.q4k is not None else 0)


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


def prepare_q8_0(W: torch.Tensor, bias: torch.Tensor | None) -> PreparedLinear:
    """Encode W once (offline) as GGUF Q8_0: 8.5 bits per weight."""
    N, K = W.shape
    qs, d = ops.q8_0_quantize(W)
    return PreparedLinear(False, N, K, bias, q8_qs=qs, q8_d=d)


def prepare_q4_k(W: torch.Tensor, bias: torch.Tensor | None) -> PreparedLinear:
    """Encode W once (offline) as GGUF Q4_K: 4-bit codes in super-blocks of
    256 (4.5 bits per weight)."""
    N, K = W.shape
    return PreparedLinear(False, N, K, bias, q4k=ops.q4_k_quantize(W))


class Workspace:
    """Reusable buffers (Xq, x_scale, and the decoded bf16 weights of a GGUF
    layer) so that a forward allocates nothing once the largest shape has
    been seen."""

    def __init__(self, device):
        self.device = device
        self._xq = None
        self._xs = None
        self._wd = None

    def weights(self, N: int, K: int) -> torch.Tensor:
        if self._wd is None or self._wd.numel() < N * K:
            self._wd = torch.empty(N * K, dtype=torch.bfloat16, device=self.device)
        return self._wd[: N * K].view(N, K)

    def get(self, M: int, K: int):
        need = M * K
        if self._xq is None or self._xq.numel() < need:
            self._xq = torch.empty(need, dtype=torch.int8, device=self.device)
        if self._xs is None or self._xs.numel() < M:
            self._xs = torch.empty(M, dtype=torch.float32, device=self.device)
        return self._xq[:need].view(M, K), self._xs[:M]


def route(layer: PreparedLinear, X: torch.Tensor, out: torch.Tensor | None = None,
          ws: Workspace | None = None) -> torch.Tensor:
    """Y = layer(X): bf16_linear for a protected layer, the weight-only
    linear for a Q8_0 or Q4_K layer, else quant + W8A8 GEMM."""
    if layer.protected:
        return ops.bf16_linear(X, layer.W, layer.bias, out=out)
    if layer.q8_0:
        work = ws.weights(layer.N, layer.K) if ws is not None else None
        return ops.q8_0_linear(X, layer.q8_qs, layer.q8_d, layer.bias, work=work, out=out)
    if layer.q4k is not None:
        work = ws.weights(layer.N, layer.K) if ws is not None else None
        return ops.q4_k_linear(X, layer.q4k, layer.bias, work=work, out=out)
    M = X.shape[0]
    if ws is None:
        Xq = x_scale = None
    else:
        Xq, x_scale = ws.get(M, layer.K)
    Xq, x_scale = ops.w8a8_quant_act(X, layer.inv_lambda, Xq=Xq, x_scale=x_scale)
    return ops.w8a8_linear(Xq, x_scale, layer.Wq, layer.w_scale, layer.bias, out=out)


def route_modulated(layer: PreparedLinear, X: torch.Tensor, shift: torch.Tensor,
                    scale: torch.Tensor, eps: float = 1e-6, out: torch.Tensor | None = None,
                    ws: Workspace | None = None) -> torch.Tensor:
    """Y = layer(bf16(LayerNorm(X) * (1 + scale) + shift)) for a W8A8 layer
    whose input a DiT block modulates (QKV, FFN up): the modulation fused
    into the activation quantization (w8a8_adaln_quant_act), then the W8A8
    GEMM. The fused step feeds the W8A8 path only; protected and GGUF layers
    raise (in a DiT their inputs are not modulated)."""
    if layer.protected or layer.weight_only:
        raise ValueError("route_modulated takes W8A8 layers only; the fused adaLN step feeds "
                         "the INT8 path")
    M = X.shape[0]
    if ws is None:
        Xq = x_scale = None
    else:
        Xq, x_scale = ws.get(M, layer.K)
    Xq, x_scale = ops.w8a8_adaln_quant_act(X, shift, scale, layer.inv_lambda, eps, Xq=Xq,
                                           x_scale=x_scale)
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
