"""The hot path under HIP graph capture: activation quantization, the W8A8
linear and the protected bf16 linear enqueue no allocation and no memset, so
one step of them can be captured once and replayed. Each replay, with eager
work and synchronizations between replays, must give the eager results bit
for bit (the persistent, two-slot and warp-specialized GEMM kernels, and
the adaLN-fused step)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import synth
from paper_2606_12280_amd import layer, ops

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(synth.to_bf16_bits(a)).view(np.int16)).to(
        DEV).view(torch.bfloat16)


@pytest.mark.parametrize("M,N,K", [(2000, 16384, 512), (4608, 4096, 1024), (1000, 4096, 1024)])
def test_captured_step_replays_bit_identical(M, N, K):
    print(f"graph capture M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng([190, M, N, K])
    X = _bf16(synth.outlier_activations(rng, M, K, K // 100, 20.0))
    W = _bf16(rng.normal(0, 0.02, (N, K)).astype(np.float32))
    b = _bf16(rng.normal(0, 0.01, N).astype(np.float32))
    sh = _bf16(rng.normal(0, 0.05, K).astype(np.float32))
    sc = _bf16(rng.normal(0, 0.1, K).astype(np.float32))
    s = torch.zeros(K, dtype=torch.float32, device=DEV)
    ops.w8a8_act_absmax(X, s)
    lam = ops.w8a8_smooth_factors(s, W, 0.5)
    lin = layer.prepare_linear(W, b, lam, protected=False)
    prot = layer.prepare_linear(W, b, None, protected=True)

    Xq = torch.empty(M, K, dtype=torch.int8, device=DEV)
    xs = torch.empty(M, dtype=torch.float32, device=DEV)
    Xq2 = torch.empty_like(Xq)
    xs2 = torch.empty_like(xs)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device=DEV)
    Y2 = torch.empty_like(Y)
    Yb = torch.empty_like(Y)

    def step():
        ops.w8a8_quant_act(X, lin.inv_lambda, Xq=Xq, x_scale=xs)
        ops.w8a8_linear(Xq, xs, lin.Wq, lin.w_scale, lin.bias, out=Y)
        ops.w8a8_adaln_quant_act(X, sh, sc, lin.inv_lambda, Xq=Xq2, x_scale=xs2)
        ops.w8a8_linear(Xq2, xs2, lin.Wq, lin.w_scale, lin.bias, out=Y2)
        ops.bf16_linear(X, prot.W, prot.bias, out=Yb)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (Xq, xs, Y, Xq2, xs2, Y2, Yb)]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for t in (Xq, xs, Y, Xq2, xs2, Y2, Yb):
            t.zero_()
        junk = (X.float() * 2).sum()  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        for name, t, r in zip(("Xq", "x_scale", "Y", "adaLN Xq", "adaLN x_scale", "adaLN Y", "bf16 Y"),
                              (Xq, xs, Y, Xq2, xs2, Y2, Yb), ref):
            assert torch.equal(t.view(torch.uint8), r.view(torch.uint8)), (rep, name)
