"""Several host threads calling the library at once, each on its own stream
and tensors (the library keeps per-device launch facts in atomics): every
output equals the same call made alone, bit for bit. The no-allocation
moments call shares one device array by design and is not called here."""
from __future__ import annotations

import threading

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


def _case(seed, M, N, K):
    rng = np.random.default_rng(seed)
    X = _bf16(synth.outlier_activations(rng, M, K, max(1, K // 100), 20.0))
    W = _bf16(rng.normal(0, 0.02, (N, K)).astype(np.float32))
    b = _bf16(rng.normal(0, 0.01, N).astype(np.float32))
    sh = _bf16(rng.normal(0, 0.05, K).astype(np.float32))
    sc = _bf16(rng.normal(0, 0.1, K).astype(np.float32))
    s = torch.zeros(K, dtype=torch.float32, device=DEV)
    ops.w8a8_act_absmax(X, s)
    lin = layer.prepare_linear(W, b, ops.w8a8_smooth_factors(s, W, 0.5), protected=False)
    return X, sh, sc, lin


def _work(X, sh, sc, lin):
    Y = layer.route(lin, X)
    Y2 = layer.route_modulated(lin, X, sh, sc)
    st = ops.w8a8_act_moments(X)
    return [Y.view(torch.int16), Y2.view(torch.int16), st.view(torch.int64)]


def test_concurrent_host_threads_match_sequential_calls():
    print("4 host threads, own streams: route, route_modulated, moments", flush=True)
    shapes = [(1000, 4096, 4096), (2304, 2048, 1024), (777, 1536, 8192), (4608, 4096, 512)]
    cases = [_case([200, i], *shp) for i, shp in enumerate(shapes)]
    ref = [_work(*c) for c in cases]
    torch.cuda.synchronize()
    out = [None] * len(cases)
    errors = []

    def run(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(3):
                    r = _work(*cases[i])
                s.synchronize()
            out[i] = r
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    assert all(not t.is_alive() for t in threads)
    for i, (a, b) in enumerate(zip(out, ref)):
        for j, (x, y) in enumerate(zip(a, b)):
            assert torch.equal(x, y), (i, j)
