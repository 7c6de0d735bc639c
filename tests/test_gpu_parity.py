"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
the same seeded inputs.

Bit-exact: inv_lambda, Wq, w_scale, Xq, x_scale, the int32 accumulators and
the calibration absmax. Within the stated tolerance: the W8A8 bf16 output
(<= 2 bf16 ulp, binary32 floor under cancellation), lambda (<= 1 binary32
ulp) and the protected bf16 output (binary64 reference with the binary32
summation bound). Full-size workloads are checked on whole tensors, the
int32 accumulators and the W8A8 output included; the protected output there
on sampled token rows."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth
from bf16ref import bf16_to_f64
from parity import (DEV, check_bf16_output, check_w8a8_output, dev, dev_bf16, host,
                    host_bits)

pytestmark = pytest.mark.gpu

from paper_2606_12280_amd import ops  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _setup():
    oracle.build()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    yield
    torch.cuda.synchronize()


def _quant_case(X, lam, M, K):
    """GPU and oracle quantization of X with smoothing lam; returns both."""
    il_ref = (1.0 / lam.astype(np.float64)).astype(np.float32)
    Xq_ref, xs_ref = oracle.quant_act(X, il_ref, M, K)
    Xq, xs = ops.w8a8_quant_act(dev_bf16(X.reshape(M, K)), dev(il_ref))
    return host(Xq), host(xs), Xq_ref, xs_ref


# --------------------------------------------------------------------------
# quantization kernels
# --------------------------------------------------------------------------

@pytest.mark.parametrize("M,K", [(1, 64), (5, 192), (64, 256), (33, 512), (7, 1088),
                                 (19, 2048), (64, 4096), (3, 4160), (9, 8192),
                                 (4, 12352), (3, 16384), (2, 32768), (1, 65536)])
def test_quant_act_bit_exact(M, K):
    c = synth.linear_case([100, M, K], M, 8, K, act="gelu")
    rng = np.random.default_rng([101, K])
    lam = np.exp(rng.uniform(-2, 2, K)).astype(np.float32)
    Xq, xs, Xq_ref, xs_ref = _quant_case(c["X"], lam, M, K)
    assert np.array_equal(xs, xs_ref)
    assert np.array_equal(Xq, Xq_ref)


@pytest.mark.parametrize("M,K", [(300001, 64), (65537, 1024), (20011, 4096), (3001, 16384)])
def test_quant_act_many_rows_per_group(M, K):
    """Long inputs: one launch holds as many row groups as the GPU keeps
    resident and each walks dozens of rows, the last of them ragged; every
    code and scale bit-exact."""
    rng = np.random.default_rng([102, M, K])
    X = synth.to_bf16_bits(synth.outlier_activations(rng, M, K, max(1, K // 100), 20.0))
    lam = np.exp(rng.uniform(-2, 2, K)).astype(np.float32)
    Xq, xs, Xq_ref, xs_ref = _quant_case(X, lam, M, K)
    assert np.array_equal(xs, xs_ref)
    assert np.array_equal(Xq, Xq_ref)


def test_quant_act_special_rows():
    """Zero, tiny (below 2^-96), constant, one-hot and tie rows, a row of
    binary32 subnormals (its absmax too is a subnormal bit pattern) and a
    row of negative zeros."""
    K = 256
    rows = np.zeros((8, K), np.float32)
    rows[1, :] = -3.0
    rows[2, :] = 2.0 ** -100
    rows[3, 17] = 0.375
    rows[4, :16] = [127.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5, 126.5, -126.5,
                    0.25, 0.75, -0.75, 64.5, 65.5, 0.0]
    rows[5, :] = np.linspace(-1e-20, 1e-20, K)
    rows[6, :] = np.ldexp(np.arange(1, K + 1, dtype=np.float32), -140) * (-1) ** np.arange(K)
    rows[7, :] = -0.0
    X = synth.to_bf16_bits(rows)
    Xq, xs, Xq_ref, xs_ref = _quant_case(X, np.ones(K, np.float32), 8, K)
    assert np.array_equal(xs, xs_ref) and np.array_equal(Xq, Xq_ref)
    for r in (0, 2, 6, 7):
        assert xs[r] == 0 and not Xq[r].any()


@pytest.mark.parametrize("N,K", [(512, 256), (100, 4096), (33, 16384), (7, 1024)])
def test_prepare_weight_bit_exact(N, K):
    c = synth.linear_case([102, N, K], 4, N, K)
    rng = np.random.default_rng([103, K])
    lam = np.exp(rng.uniform(-3, 3, K)).astype(np.float32)
    Wq_ref, ws_ref, il_ref = oracle.prepare_weight(c["W"], lam, N, K)
    Wq, ws, il = ops.w8a8_prepare_weight(dev_bf16(c["W"]), dev(lam))
    assert np.array_equal(host(il), il_ref)
    assert np.array_equal(host(ws), ws_ref)
    assert np.array_equal(host(Wq), Wq_ref)


@pytest.mark.parametrize("M,K", [(64, 256), (4608, 4096), (1000, 16384), (3, 64), (77, 384),
                                 (300, 1088)])
def test_act_absmax_bit_exact_and_accumulates(M, K):
    X1 = synth.rand_bf16([104, M, K], (M, K), 2.0)
    X2 = synth.rand_bf16([105, M, K], (7, K), 5.0)
    ref = oracle.act_absmax(X2, 7, K, oracle.act_absmax(X1, M, K))
    s = torch.zeros(K, dtype=torch.float32, device="cuda")
    ops.w8a8_act_absmax(dev_bf16(X1), s)
    ops.w8a8_act_absmax(dev_bf16(X2), s)
    assert np.array_equal(host(s), ref)


@pytest.mark.parametrize("alpha", [0.5, 0.3])
def test_smooth_factors(alpha):
    c = synth.tiny_case()
    M, N, K = c["M"], c["N"], c["K"]
    s_ref = oracle.act_absmax(c["X"], M, K)
    s_ref[5] = 0.0                              # lambda = 1 rule
    lam_ref = oracle.smooth_factors(s_ref, c["W"], N, K, alpha)
    lam = host(ops.w8a8_smooth_factors(dev(s_ref), dev_bf16(c["W"]), alpha))
    assert lam[5] == 1.0
    ulps = np.abs(lam.view(np.int32).astype(np.int64) - lam_ref.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1
    if alpha == 0.5:
        assert np.array_equal(lam, lam_ref)     # sqrt and divide are correctly rounded


# --------------------------------------------------------------------------
# fragility profile (Section 3, "Activation-fragility profiling and
# protection")
# --------------------------------------------------------------------------

def _check_moments(got, ref):
    """max |x| bit-exact; mean, std and kurtosis to binary64 summation-order
    error (the GPU adds in a different order than the oracle)."""
    assert got[0] == ref[0]
    assert abs(got[1] - ref[1]) <= 1e-13 * ref[2] + 1e-15 * abs(ref[1])
    assert got[2] == pytest.approx(ref[2], rel=1e-12)
    assert got[3] == pytest.approx(ref[3], rel=1e-10)


@pytest.mark.parametrize("M,K,act", [(1, 64, "normal"), (3, 192, "gelu"), (257, 1088, "gelu"),
                                     (64, 4096, "outlier"), (1000, 16384, "gelu")])
def test_act_moments_parity(M, K, act):
    c = synth.linear_case([115, M, K], M, 8, K, act=act)
    ref = oracle.act_moments(c["X"], M, K)
    got = host(ops.w8a8_act_moments(dev_bf16(c["X"])))
    _check_moments(got, ref)


def test_act_moments_special_inputs():
    """Constant input (std 0, kurtosis 0), +-a (kurtosis exactly 1), a single
    outlier entry, and the largest bf16 magnitudes."""
    two = synth.to_bf16_bits(np.array([0.75, -0.75], np.float32))
    big = synth.to_bf16_bits(np.array([3.0e38, -3.0e38], np.float32))
    cases = [np.full((5, 64), 0x4040, np.uint16), np.tile(two, (7, 64)),
             np.tile(big, (2, 64))]
    one = np.zeros((9, 128), np.uint16)
    one[4, 77] = 0x4480                                  # 1024.0
    cases.append(one)
    for X in cases:
        M, K = X.shape
        ref = oracle.act_moments(X, M, K)
        got = host(ops.w8a8_act_moments(dev_bf16(X)))
        if ref[2] == 0.0:
            assert list(got) == list(ref)
        else:
            _check_moments(got, ref)
    assert list(host(ops.w8a8_act_moments(dev_bf16(np.tile(two, (7, 64)))))) == [0.75, 0.0, 0.75, 1.0]


def test_act_moments_full_size_and_deterministic():
    c = synth.ffn_down_case()
    X = dev_bf16(c["X"])
    ref = oracle.act_moments(c["X"], c["M"], c["K"])
    work = torch.empty(_lib_work_bytes(), dtype=torch.uint8, device=DEV)
    a = host(ops.w8a8_act_moments(X, work))
    b = host(ops.w8a8_act_moments(X, work))
    assert np.array_equal(a, b)                          # same bits on every call
    _check_moments(a, ref)


def test_profile_selects_like_the_oracle():
    """A 6-layer, 3-step profile through fragility.Profile: the selected
    layers equal the oracle's top-2 of the oracle's own statistics."""
    from paper_2606_12280_amd import fragility
    L, T, M, K = 6, 3, 64, 256
    prof = fragility.Profile(L, T, DEV)
    kurt = np.zeros((L, T))
    for layer in range(L):
        for step in range(T):
            act = "gelu" if layer in (1, 4) else "normal"
            c = synth.linear_case([116, layer, step], M, 8, K, act=act)
            prof.record(layer, step, dev_bf16(c["X"]))
            kurt[layer, step] = oracle.act_moments(c["X"], M, K)[3]
    table = prof.table()
    assert np.allclose(table[:, :, 3], kurt, rtol=1e-10)
    want = oracle.top_n(oracle.fragility_scores(kurt), 2)
    assert fragility.select_protected(prof.scores(), 2) == want
    assert sorted(want) == [1, 4]


def _lib_work_bytes():
    from paper_2606_12280_amd import _lib
    return _lib.MOMENTS_WORK_BYTES


# --------------------------------------------------------------------------
# GEMMs on small and ragged shapes (full outputs)
# --------------------------------------------------------------------------

GEMM_SHAPES = [(1, 1, 64), (64, 512, 256), (257, 129, 192), (300, 520, 1088),
               (513, 384, 4160), (31, 1000, 64), (256, 128, 128), (200, 4096, 512)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_i32_bit_exact(M, N, K):
    A = synth.rand_i8([106, M, K], (M, K))
    B = synth.rand_i8([107, N, K], (N, K))
    ref = oracle.gemm_i32(A, B, M, N, K)
    C = host(ops.w8a8_gemm_i32(dev(A), dev(B)))
    assert np.array_equal(C, ref)


# Shapes large enough to select the two-slot kernels (288 x 256 tiles, and
# 192 x 256 for the third), with ragged M and N (N odd: element stores at
# the edge) and 1, 2, 3 and 5 K tiles of 128 bytes.
LARGE_RAGGED = [(4571, 16376, 128), (4600, 16375, 256), (4545, 12290, 384),
                (4608, 16384, 640)]

# One ragged shape per GEMM configuration, with the (tile_m, tile_n,
# threads) the library reports for it.
CONFIG_SHAPES = [
    ((4571, 16376, 128), (288, 256, 768)),
    ((4545, 4350, 384), (192, 256, 512)),
    ((250, 1000, 256), (192, 128, 512)),
    ((1000, 8190, 256), (256, 128, 512)),
    ((513, 384, 4160), (192, 256, 256)),
]


@pytest.mark.parametrize("shape,config", CONFIG_SHAPES)
def test_every_gemm_configuration(shape, config):
    """Each kernel configuration on a shape ragged in M and N: int32
    accumulators bit-exact, the dequantizing epilogue without a bias within
    tolerance, and bf16_linear within its bound on sampled rows (its rows
    have twice the bytes, so its configuration can differ)."""
    M, N, K = shape
    assert ops.w8a8_gemm_config(M, N, K) == config
    A = synth.rand_i8([116, M, K], (M, K))
    B = synth.rand_i8([117, N, K], (N, K))
    ref = oracle.gemm_i32(A, B, M, N, K)
    Ad, Bd = dev(A), dev(B)
    assert np.array_equal(host(ops.w8a8_gemm_i32(Ad, Bd)), ref)
    rng = np.random.default_rng([118, M, N, K])
    xs = rng.uniform(1e-3, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    zero = np.zeros(N, np.uint16)
    Y = host_bits(ops.w8a8_linear(Ad, dev(xs), Bd, dev(ws), None))
    check_w8a8_output(Y, oracle.epilogue(ref, xs, ws, zero, M, N), ref, xs, ws, zero)
    c = synth.linear_case([119, M, N, K], M, N, K)
    Yb = host_bits(ops.bf16_linear(dev_bf16(c["X"]), dev_bf16(c["W"]), dev_bf16(c["bias"])))
    rows = np.sort(np.concatenate([[0, M - 1], rng.choice(M, min(M, 40), replace=False)]))
    check_bf16_output(Yb[rows], c["X"].reshape(M, K)[rows], c["W"].reshape(N, K), c["bias"])


@pytest.mark.parametrize("M,N,K", LARGE_RAGGED)
def test_gemm_i32_large_ragged(M, N, K):
    A = synth.rand_i8([109, M, K], (M, K))
    B = synth.rand_i8([110, N, K], (N, K))
    ref = oracle.gemm_i32(A, B, M, N, K)
    C = host(ops.w8a8_gemm_i32(dev(A), dev(B)))
    assert np.array_equal(C, ref)


@pytest.mark.parametrize("M,N,K", LARGE_RAGGED)
@pytest.mark.parametrize("with_bias", [True, False])
def test_w8a8_linear_large_ragged(M, N, K, with_bias):
    """The dequantizing epilogue (rows staged through LDS) on whole outputs."""
    A = synth.rand_i8([111, M, K], (M, K))
    B = synth.rand_i8([112, N, K], (N, K))
    rng = np.random.default_rng([113, M, N, K])
    xs = rng.uniform(1e-3, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    b = synth.rand_bf16([114, N], (N,), 0.5) if with_bias else np.zeros(N, np.uint16)
    acc = oracle.gemm_i32(A, B, M, N, K)
    Yref = oracle.epilogue(acc, xs, ws, b, M, N)
    Y = ops.w8a8_linear(dev(A), dev(xs), dev(B), dev(ws), dev_bf16(b) if with_bias else None)
    check_w8a8_output(host_bits(Y), Yref, acc, xs, ws, b)


# Shapes that take the persistent 288 x 256 kernel (more tiles than CUs, N a
# multiple of 8, at least three 128-byte K tiles): ragged M with the fewest
# K tiles it runs (3), a tile count between one and two rounds (418 tiles,
# ragged in both M and N: some workgroups walk two tiles, the others one),
# and a long row of tiles.
PERSISTENT_SHAPES = [(4571, 16376, 384), (3163, 9720, 1024), (2000, 16384, 512),
                     (576, 131072, 384)]


@pytest.mark.parametrize("M,N,K", PERSISTENT_SHAPES)
def test_persistent_gemm_whole_outputs(M, N, K):
    """The persistent kernel on whole outputs: int32 accumulators bit-exact,
    the dequantizing epilogue with and without a bias within tolerance, and
    bf16_linear (also persistent here) within its bound on sampled rows."""
    assert ops.w8a8_gemm_config(M, N, K) == (288, 256, 768)
    A = synth.rand_i8([120, M, K], (M, K))
    B = synth.rand_i8([121, N, K], (N, K))
    acc = oracle.gemm_i32(A, B, M, N, K)
    Ad, Bd = dev(A), dev(B)
    assert np.array_equal(host(ops.w8a8_gemm_i32(Ad, Bd)), acc)
    rng = np.random.default_rng([122, M, N, K])
    xs = rng.uniform(1e-3, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    b = synth.rand_bf16([123, N], (N,), 0.5)
    zero = np.zeros(N, np.uint16)
    Y = host_bits(ops.w8a8_linear(Ad, dev(xs), Bd, dev(ws), dev_bf16(b)))
    check_w8a8_output(Y, oracle.epilogue(acc, xs, ws, b, M, N), acc, xs, ws, b)
    Y0 = host_bits(ops.w8a8_linear(Ad, dev(xs), Bd, dev(ws), None))
    check_w8a8_output(Y0, oracle.epilogue(acc, xs, ws, zero, M, N), acc, xs, ws, zero)
    del acc, Y, Y0
    c = synth.linear_case([124, M, N, K], M, N, K)
    Yb = host_bits(ops.bf16_linear(dev_bf16(c["X"]), dev_bf16(c["W"]), dev_bf16(c["bias"])))
    rows = np.unique(np.concatenate([[0, M - 1], np.arange(0, M, 288),
                                     rng.choice(M, min(M, 32), replace=False)]))
    check_bf16_output(Yb[rows], c["X"].reshape(M, K)[rows], c["W"].reshape(N, K), c["bias"])


@pytest.mark.parametrize("K", [16384, 65536])
def test_gemm_i32_extremes(K):
    """All +-127 codes: |acc| = 127^2 K, the largest sum (1.06e9 at the
    largest K the entry points accept, inside int32)."""
    M, N = 64, 96
    A = np.full((M, K), 127, np.int8)
    A[1::2] = -127
    B = np.full((N, K), -127, np.int8)
    B[::3, ::2] = 127
    C = host(ops.w8a8_gemm_i32(dev(A), dev(B)))
    assert np.array_equal(C, oracle.gemm_i32(A, B, M, N, K))
    assert abs(int(C[0, 1])) == 127 * 127 * K


def test_gemm_i32_extremes_on_the_large_tiles():
    """The same +-127 codes through the 12-wave 288 x 256 kernel (16 x 16
    MFMA blocks) at a full DiT output, 4608 x 4096, with K = 32768: every
    accumulator is +-127^2 K or 0, which the structure of the codes gives in
    closed form (A's row m is 127 s_m, s_m = +-1; B's rows n % 3 != 0 are all
    -127, the others alternate +127, -127 along K and sum to 0)."""
    M, N, K = 4608, 4096, 32768
    assert ops.w8a8_gemm_config(M, N, K) == (288, 256, 768)
    A = np.full((M, K), 127, np.int8)
    A[1::2] = -127
    B = np.full((N, K), -127, np.int8)
    B[::3, ::2] = 127
    C = host(ops.w8a8_gemm_i32(dev(A), dev(B)))
    sign = np.where(np.arange(M) % 2 == 0, 1, -1).astype(np.int64)
    rowsum_b = np.where(np.arange(N) % 3 == 0, 0, -127 * K).astype(np.int64)
    want = (127 * sign)[:, None] * rowsum_b[None, :]
    assert np.array_equal(C.astype(np.int64), want)
    assert abs(int(C[0, 1])) == 127 * 127 * K


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES + [(64, 512, 256)])
@pytest.mark.parametrize("with_bias", [True, False])
def test_w8a8_linear_recipe(M, N, K, with_bias):
    """Whole recipe through the library: prepare, quantize, linear; every
    intermediate bit-exact and Y within tolerance of the oracle."""
    c = synth.linear_case([108, M, N, K], M, N, K, bias=with_bias)
    lam = oracle.smooth_factors(oracle.act_absmax(c["X"], M, K), c["W"], N, K, 0.5)
    r = oracle.recipe(c["X"], c["W"], c["bias"], M, N, K, lam=lam)
    Wq, ws, il = ops.w8a8_prepare_weight(dev_bf16(c["W"]), dev(lam))
    Xq, xs = ops.w8a8_quant_act(dev_bf16(c["X"]), il)
    bias = dev_bf16(c["bias"]) if with_bias else None
    Y = ops.w8a8_linear(Xq, xs, Wq, ws, bias)
    C = ops.w8a8_gemm_i32(Xq, Wq)
    assert np.array_equal(host(Wq), r["Wq"]) and np.array_equal(host(ws), r["w_scale"])
    assert np.array_equal(host(Xq), r["Xq"]) and np.array_equal(host(xs), r["x_scale"])
    assert np.array_equal(host(C), r["acc"])
    check_w8a8_output(host_bits(Y), r["Y"], r["acc"], r["x_scale"], r["w_scale"], c["bias"])


def test_w8a8_linear_tiny_case_and_determinism():
    c = synth.tiny_case()
    M, N, K = c["M"], c["N"], c["K"]
    r = oracle.recipe(c["X"], c["W"], c["bias"], M, N, K)
    Wq, ws, il = ops.w8a8_prepare_weight(dev_bf16(c["W"]), dev(r["lambda"]))
    Xq, xs = ops.w8a8_quant_act(dev_bf16(c["X"]), il)
    Y1 = host_bits(ops.w8a8_linear(Xq, xs, Wq, ws, dev_bf16(c["bias"])))
    Y2 = host_bits(ops.w8a8_linear(Xq, xs, Wq, ws, dev_bf16(c["bias"])))
    assert np.array_equal(Y1, Y2)
    mx, eq = check_w8a8_output(Y1, r["Y"], r["acc"], r["x_scale"], r["w_scale"], c["bias"])
    assert eq > 0.9


def test_outputs_stay_inside_their_bounds():
    """Guard bands around ragged outputs: no store lands outside Y or C."""
    M, N, K = 257, 129, 192
    A = synth.rand_i8([109], (M, K))
    B = synth.rand_i8([110], (N, K))
    pad = 4096
    Cbuf = torch.full((M * N + 2 * pad,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    C = Cbuf[pad:pad + M * N].view(M, N)
    ops.w8a8_gemm_i32(dev(A), dev(B), out=C)
    Cb = host(Cbuf)
    assert np.all(Cb[:pad] == 0x5A5A5A5A) and np.all(Cb[pad + M * N:] == 0x5A5A5A5A)
    Ybuf = torch.full((M * N + 2 * pad,), 0x1234, dtype=torch.int16, device="cuda")
    Y = Ybuf[pad:pad + M * N].view(torch.bfloat16).view(M, N)
    xs = dev(np.ones(M, np.float32))
    ws = dev(np.ones(N, np.float32))
    ops.w8a8_linear(dev(A), xs, dev(B), ws, None, out=Y)
    ops.bf16_linear(dev_bf16(synth.rand_bf16(1, (M, K))), dev_bf16(synth.rand_bf16(2, (N, K))),
                    None, out=Y)
    Yb = host(Ybuf)
    assert np.all(Yb[:pad] == 0x1234) and np.all(Yb[pad + M * N:] == 0x1234)


def test_nondefault_stream():
    M, N, K = 130, 260, 320
    A = synth.rand_i8([111], (M, K))
    B = synth.rand_i8([112], (N, K))
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        C = ops.w8a8_gemm_i32(dev(A), dev(B))
    s.synchronize()
    assert np.array_equal(host(C), oracle.gemm_i32(A, B, M, N, K))


# --------------------------------------------------------------------------
# protected bf16 path
# --------------------------------------------------------------------------

@pytest.mark.parametrize("M,N,K", [(64, 512, 256), (257, 129, 192), (100, 300, 4160),
                                   (33, 64, 16384), (4600, 4093, 256)])
def test_bf16_linear_small_integers_exact(M, N, K):
    """Integer inputs keep every binary32 partial sum exact, so the result
    must equal the oracle's bit for bit (catches any dropped or repeated
    K block). The last shape runs the 12-wave 288 x 256 kernel with an odd N,
    whose rows go out element by element."""
    rng = np.random.default_rng([113, M, N, K])
    X = synth.to_bf16_bits(rng.integers(-8, 9, (M, K)).astype(np.float32))
    W = synth.to_bf16_bits(rng.integers(-8, 9, (N, K)).astype(np.float32))
    b = synth.to_bf16_bits(rng.integers(-64, 64, N).astype(np.float32))
    Y = host_bits(ops.bf16_linear(dev_bf16(X), dev_bf16(W), dev_bf16(b)))
    assert np.array_equal(Y, oracle.bf16_linear(X, W, b, M, N, K))


@pytest.mark.parametrize("M,N,K", [(64, 512, 256), (300, 520, 1088), (65, 128, 16384),
                                   (4571, 16376, 192), (33, 70, 65536)])
def test_bf16_linear_random(M, N, K):
    c = synth.linear_case([114, M, N, K], M, N, K, act="gelu")
    Y = host_bits(ops.bf16_linear(dev_bf16(c["X"]), dev_bf16(c["W"]), dev_bf16(c["bias"])))
    check_bf16_output(Y, c["X"].reshape(M, K), c["W"].reshape(N, K), c["bias"])
    ref = oracle.bf16_linear(c["X"], c["W"], c["bias"], M, N, K)
    from bf16ref import ulp_distance
    assert (ulp_distance(Y, ref) <= 1).mean() > 0.999


# --------------------------------------------------------------------------
# full-size DiT workloads, whole tensors: the codes and scales, the int32
# accumulators of every token row and output channel, and the bf16 output,
# in the launch configuration the benchmark times
# --------------------------------------------------------------------------

PROTECTED_SAMPLE_ROWS = 64


def _full_size_check(c, protected_too=False):
    M, N, K = c["M"], c["N"], c["K"]
    lam = oracle.smooth_factors(oracle.act_absmax(c["X"], M, K), c["W"], N, K, 0.5)
    Wq_ref, ws_ref, il_ref = oracle.prepare_weight(c["W"], lam, N, K)
    Xq_ref, xs_ref = oracle.quant_act(c["X"], il_ref, M, K)
    Xd, Wd = dev_bf16(c["X"].reshape(M, K)), dev_bf16(c["W"].reshape(N, K))
    bd = dev_bf16(c["bias"])
    s = torch.zeros(K, dtype=torch.float32, device="cuda")
    ops.w8a8_act_absmax(Xd, s)
    lam_gpu = ops.w8a8_smooth_factors(s, Wd, 0.5)
    assert np.array_equal(host(lam_gpu), lam)
    Wq, ws, il = ops.w8a8_prepare_weight(Wd, dev(lam))
    Xq, xs = ops.w8a8_quant_act(Xd, il)
    assert np.array_equal(host(il), il_ref)
    assert np.array_equal(host(ws), ws_ref) and np.array_equal(host(Wq), Wq_ref)
    assert np.array_equal(host(xs), xs_ref) and np.array_equal(host(Xq), Xq_ref)
    Y = ops.w8a8_linear(Xq, xs, Wq, ws, bd)
    C = ops.w8a8_gemm_i32(Xq, Wq)
    acc_ref = oracle.gemm_i32(Xq_ref, Wq_ref, M, N, K)          # every row
    C_h = host(C)
    del C
    bad = np.argwhere(C_h != acc_ref)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first at {bad[0].tolist()}"
    del C_h
    Y_ref = oracle.epilogue(acc_ref, xs_ref, ws_ref, c["bias"], M, N)
    check_w8a8_output(host_bits(Y), Y_ref, acc_ref, xs_ref, ws_ref, c["bias"])
    del acc_ref, Y_ref
    if protected_too:
        # the protected output is order-dependent: checked against binary64
        # with the summation bound on sampled rows (first, last and a seeded
        # draw covering every 288-row tile row)
        Yb = host_bits(ops.bf16_linear(Xd, Wd, bd))
        rng = np.random.default_rng([115, M, N, K])
        rows = np.unique(np.concatenate([[0, M - 1], np.arange(0, M, 288),
                                         rng.choice(M, PROTECTED_SAMPLE_ROWS, replace=False)]))
        check_bf16_output(Yb[rows], c["X"].reshape(M, K)[rows], c["W"].reshape(N, K), c["bias"])


def test_full_size_ffn_up():
    """4608 x 4096 -> 16384 (one branch's FFN up-projection), whole output."""
    _full_size_check(synth.ffn_up_case())


def test_full_size_ffn_down_both_paths():
    """4608 x 16384 -> 4096 with post-GELU heavy-tailed activations, W8A8 on
    the whole output and the protected bf16 path."""
    _full_size_check(synth.ffn_down_case(), protected_too=True)


@pytest.mark.parametrize("branch", [0, 1])
def test_full_size_dit_block(branch):
    """The four linears of one DiT block for one CFG branch through the
    router: the three W8A8 linears on whole tensors (codes, scales, int32
    accumulators, bf16 output), the FFN down routed to the protected path."""
    from paper_2606_12280_amd import layer as L
    ws = L.Workspace(DEV)
    for li in range(4):
        c = synth.block_case(branch, li)
        M, N, K = c["M"], c["N"], c["K"]
        lam = oracle.smooth_factors(oracle.act_absmax(c["X"], M, K), c["W"], N, K, 0.5)
        protected = c["name"] == "ffn_down"
        Xd, Wd = dev_bf16(c["X"].reshape(M, K)), dev_bf16(c["W"].reshape(N, K))
        lay = L.prepare_linear(Wd, dev_bf16(c["bias"]), dev(lam), protected)
        Y = host_bits(L.route(lay, Xd, ws=ws))
        if protected:
            rows = np.unique(np.concatenate([
                np.arange(0, M, 288), np.random.default_rng([116, branch, li]).choice(M, 16, replace=False)]))
            check_bf16_output(Y[rows], c["X"].reshape(M, K)[rows], c["W"].reshape(N, K),
                              c["bias"])
            continue
        Wq_ref, ws_ref, il_ref = oracle.prepare_weight(c["W"], lam, N, K)
        assert np.array_equal(host(lay.Wq), Wq_ref) and np.array_equal(host(lay.w_scale), ws_ref)
        assert np.array_equal(host(lay.inv_lambda), il_ref)
        Xq_ref, xs_ref = oracle.quant_act(c["X"], il_ref, M, K)
        Xq, xs = ops.w8a8_quant_act(Xd, lay.inv_lambda)
        assert np.array_equal(host(Xq), Xq_ref) and np.array_equal(host(xs), xs_ref)
        acc = oracle.gemm_i32(Xq_ref, Wq_ref, M, N, K)
        C = host(ops.w8a8_gemm_i32(Xq, lay.Wq))
        bad = np.argwhere(C != acc)
        assert bad.size == 0, f"{c['name']}: {len(bad)} accumulators differ, first at {bad[0].tolist()}"
        del C
        Y_ref = oracle.epilogue(acc, xs_ref, ws_ref, c["bias"], M, N)
        check_w8a8_output(Y, Y_ref, acc, xs_ref, ws_ref, c["bias"])


# --------------------------------------------------------------------------
# GGUF Q8_0 weight-only (Section 3, "GGUF k-quants")
# --------------------------------------------------------------------------

def _q8_case(seed, N, K):
    W = synth.rand_bf16(seed, (N, K), 0.02)
    if N > 1 and K >= 128:                      # a zero block and a large one
        W[0, :32] = 0
        W[1, 64:96] = synth.rand_bf16([seed, 1], (32,), 40.0)
    return W


@pytest.mark.parametrize("N,K", [(1, 64), (7, 256), (33, 1088), (512, 4096)])
def test_q8_0_codes_scales_and_decode_bit_exact(N, K):
    W = _q8_case([150, N, K], N, K)
    qs_ref, d_ref = oracle.q8_0_quantize(W, N, K)
    qs, d = ops.q8_0_quantize(dev_bf16(W))
    assert np.array_equal(host(qs), qs_ref)
    assert np.array_equal(host(d).view(np.uint16), d_ref)
    Wd = ops.q8_0_dequantize(qs, d)
    assert np.array_equal(host_bits(Wd), oracle.q8_0_dequantize(qs_ref, d_ref, N, K))


def test_q8_0_special_blocks_on_gpu():
    """Zero, underflowing (scale 0) and capped (scale 65504, codes clamp)
    blocks, and round-half-even ties with scale 1."""
    W = np.zeros((2, 128), np.float32)
    W[0, 32:64] = 2.0 ** -30
    W[0, 64] = 9.0e6
    W[0, 65] = -1.0e6
    W[1, :8] = [127.0, 0.5, -0.5, 1.5, 2.5, -2.5, 3.5, 126.5]
    B = synth.to_bf16_bits(W)
    qs_ref, d_ref = oracle.q8_0_quantize(B, 2, 128)
    qs, d = ops.q8_0_quantize(dev_bf16(B))
    assert np.array_equal(host(qs), qs_ref)
    assert np.array_equal(host(d).view(np.uint16), d_ref)
    assert list(host(qs)[1, :8]) == [127, 0, 0, 2, 2, -2, 4, 126]


@pytest.mark.parametrize("M,N,K", [(64, 512, 256), (257, 129, 192), (300, 520, 1088)])
def test_q8_0_linear(M, N, K):
    c = synth.linear_case([151, M, N, K], M, N, K, act="gelu")
    qs_ref, d_ref = oracle.q8_0_quantize(c["W"], N, K)
    Wd = oracle.q8_0_dequantize(qs_ref, d_ref, N, K)
    qs, d = ops.q8_0_quantize(dev_bf16(c["W"]))
    Y = host_bits(ops.q8_0_linear(dev_bf16(c["X"]), qs, d, dev_bf16(c["bias"])))
    check_bf16_output(Y, c["X"].reshape(M, K), Wd, c["bias"])
    ref = oracle.q8_0_linear(c["X"], qs_ref, d_ref, c["bias"], M, N, K)
    from bf16ref import ulp_distance
    assert (ulp_distance(Y, ref) <= 1).mean() > 0.999


def test_q8_0_full_size_ffn_up():
    """FFN up weights 16384 x 4096: codes and scales bit-exact on the whole
    tensor; the linear on 24 sampled token rows."""
    c = synth.ffn_up_case()
    M, N, K = c["M"], c["N"], c["K"]
    qs_ref, d_ref = oracle.q8_0_quantize(c["W"], N, K)
    qs, d = ops.q8_0_quantize(dev_bf16(c["W"]))
    assert np.array_equal(host(qs), qs_ref)
    assert np.array_equal(host(d).view(np.uint16), d_ref)
    X = c["X"].reshape(M, K)
    Y = host_bits(ops.q8_0_linear(dev_bf16(X), qs, d, dev_bf16(c["bias"])))
    rows = np.random.default_rng(152).choice(M, 24, replace=False)
    Wd = oracle.q8_0_dequantize(qs_ref, d_ref, N, K)
    check_bf16_output(Y[rows], X[rows], Wd, c["bias"])


# --------------------------------------------------------------------------
# GGUF Q4_K weight-only (Section 3, "GGUF k-quants")
# --------------------------------------------------------------------------

def _q4k_case(seed, N, K):
    W = synth.rand_bf16(seed, (N, K), 0.02).reshape(N, K)
    Wf = bf16_to_f64(W).reshape(N, K).astype(np.float32)
    rng = np.random.default_rng(seed)
    Wf[:, rng.choice(K, max(1, K // 64), replace=False)] *= 12     # outlier channels
    if N >= 4:
        Wf[1] = np.abs(Wf[1])                                       # no offsets needed
        Wf[2] += 0.01                                               # a mean offset
    if K >= 512 and N >= 4:
        Wf[3, :256] = 0                                             # a zero super-block
        Wf[3, 256:288] = -0.75                                      # a constant sub-block
        Wf[3, 300] = 3.0e9                                          # d capped at 65504
    return synth.to_bf16_bits(Wf)


def _q4k_host(q):
    return {"qs": host(q.qs), "scales": host(q.scales),
            "d": host(q.d).view(np.uint16), "dmin": host(q.dmin).view(np.uint16)}


def _check_q4k_planes(q, ref):
    got = _q4k_host(q)
    for name in ("qs", "scales", "d", "dmin"):
        assert np.array_equal(got[name], ref[name]), name


@pytest.mark.parametrize("N,K", [(1, 256), (7, 512), (33, 1280), (512, 4096)])
def test_q4_k_planes_and_decode_bit_exact(N, K):
    W = _q4k_case([160, N, K], N, K)
    ref = oracle.q4_k_quantize(W, N, K)
    q = ops.q4_k_quantize(dev_bf16(W))
    _check_q4k_planes(q, ref)
    assert np.array_equal(host_bits(ops.q4_k_dequantize(q)), oracle.q4_k_dequantize(ref, N, K))


@pytest.mark.parametrize("fmt", ["q8_0", "q4_k"])
def test_gguf_decode_past_2_28_workgroups(fmt):
    """A 32832 x 65536 weight: N K / 8 decode threads need more than 2^20
    workgroups of 256, so the decode grid takes its second dimension (the
    last 64 rows). The weight is a 64-row block tiled 513 times; the first
    and last copies are checked against the oracle's decode of the block."""
    R0, K = 64, 65536
    N = 513 * R0
    assert N * K // 8 > (1 << 28)
    blk = _q8_case([170, R0, K], R0, K) if fmt == "q8_0" else _q4k_case([171, R0, K], R0, K)
    Wd = dev_bf16(blk).repeat(N // R0, 1)
    if fmt == "q8_0":
        qs_ref, d_ref = oracle.q8_0_quantize(blk, R0, K)
        ref = oracle.q8_0_dequantize(qs_ref, d_ref, R0, K)
        qs, d = ops.q8_0_quantize(Wd)
        del Wd
        out = ops.q8_0_dequantize(qs, d)
        assert np.array_equal(host(qs[-R0:]), qs_ref)
        del qs, d
    else:
        ref_planes = oracle.q4_k_quantize(blk, R0, K)
        ref = oracle.q4_k_dequantize(ref_planes, R0, K)
        q = ops.q4_k_quantize(Wd)
        del Wd
        out = ops.q4_k_dequantize(q)
        assert np.array_equal(host(q.qs[-R0:]), ref_planes["qs"])
        del q
    assert np.array_equal(host_bits(out[:R0]), ref)
    assert np.array_equal(host_bits(out[-R0:]), ref)
    del out
    torch.cuda.empty_cache()


def test_q4_k_decode_of_arbitrary_planes():
    """Decoding planes the encoder would not produce (every code, 6-bit
    value and a wide range of binary16 scales) matches the oracle."""
    rng = np.random.default_rng(161)
    N, K = 16, 1024
    packed = np.stack([oracle.q4_k_pack_scales(rng.integers(0, 64, 8), rng.integers(0, 64, 8))
                       for _ in range(N * K // 256)])
    ref = {"qs": rng.integers(0, 256, (N, K // 2)).astype(np.uint8),
           "scales": packed.reshape(N, K // 256 * 12),
           "d": rng.lognormal(-6, 3, (N, K // 256)).astype(np.float16).view(np.uint16),
           "dmin": rng.lognormal(-6, 3, (N, K // 256)).astype(np.float16).view(np.uint16)}
    q = ops.Q4K(dev(ref["qs"]), dev(ref["scales"]),
                dev(ref["d"].view(np.float16)), dev(ref["dmin"].view(np.float16)))
    assert np.array_equal(host_bits(ops.q4_k_dequantize(q)), oracle.q4_k_dequantize(ref, N, K))


@pytest.mark.parametrize("M,N,K", [(64, 512, 256), (257, 129, 512), (300, 520, 1280)])
def test_q4_k_linear(M, N, K):
    c = synth.linear_case([162, M, N, K], M, N, K, act="gelu")
    ref = oracle.q4_k_quantize(c["W"], N, K)
    Wd = oracle.q4_k_dequantize(ref, N, K)
    q = ops.q4_k_quantize(dev_bf16(c["W"]))
    _check_q4k_planes(q, ref)
    Y = host_bits(ops.q4_k_linear(dev_bf16(c["X"]), q, dev_bf16(c["bias"])))
    check_bf16_output(Y, c["X"].reshape(M, K), Wd, c["bias"])
    from bf16ref import ulp_distance
    assert (ulp_distance(Y, oracle.q4_k_linear(c["X"], ref, c["bias"], M, N, K)) <= 1).mean() > 0.999


def test_q4_k_full_size_ffn_up():
    """FFN up weights 16384 x 4096: every plane bit-exact on the whole
    tensor; the linear on 24 sampled token rows."""
    c = synth.ffn_up_case()
    M, N, K = c["M"], c["N"], c["K"]
    ref = oracle.q4_k_quantize(c["W"], N, K)
    q = ops.q4_k_quantize(dev_bf16(c["W"]))
    _check_q4k_planes(q, ref)
    X = c["X"].reshape(M, K)
    Y = host_bits(ops.q4_k_linear(dev_bf16(X), q, dev_bf16(c["bias"])))
    rows = np.random.default_rng(163).choice(M, 24, replace=False)
    check_bf16_output(Y[rows], X[rows], oracle.q4_k_dequantize(ref, N, K), c["bias"])


# --------------------------------------------------------------------------
# adaLN modulation fused into the activation quantization (Section 2: the
# modulation is generated at run time)
# --------------------------------------------------------------------------

def _adaln_inputs(seed, M, K):
    rng = np.random.default_rng(seed)
    X = rng.normal(0, 1, (M, K)).astype(np.float32)
    X[:, rng.choice(K, max(1, K // 100), replace=False)] *= 20      # outlier channels
    X[M // 2:] += rng.normal(0, 3, (M - M // 2, 1)).astype(np.float32)
    shift = rng.normal(0, 0.05, K).astype(np.float32)
    scale = rng.normal(0, 0.1, K).astype(np.float32)
    il = rng.uniform(0.25, 4.0, K).astype(np.float32)
    return synth.to_bf16_bits(X), synth.to_bf16_bits(shift), synth.to_bf16_bits(scale), il


def _check_adaln(X, shift, scale, il, M, K, eps=1e-6):
    Xq_ref, xs_ref = oracle.adaln_quant_act(X, shift, scale, il, M, K, eps)
    Xq, xs = ops.w8a8_adaln_quant_act(dev_bf16(X), dev_bf16(shift), dev_bf16(scale), dev(il), eps)
    assert np.array_equal(host(xs).view(np.uint32), xs_ref.view(np.uint32))
    assert np.array_equal(host(Xq), Xq_ref)


@pytest.mark.parametrize("M,K", [(1, 64), (5, 256), (33, 1088), (300, 2112), (257, 4096),
                                 (64, 8192)])
def test_adaln_quant_act_bit_exact(M, K):
    _check_adaln(*_adaln_inputs([180, M, K], M, K), M, K)


@pytest.mark.parametrize("M,K", [(200003, 64), (30011, 1024), (9001, 4096), (6007, 8192)])
def test_adaln_quant_act_many_rows_per_group(M, K):
    """Long inputs: each resident row group walks dozens of rows, the last of
    them ragged; codes and scales bit-exact."""
    _check_adaln(*_adaln_inputs([183, M, K], M, K), M, K)


def test_adaln_quant_act_special_rows():
    """Constant rows (the norm is 0, so they code bf16(shift)), all-zero rows
    with zero shift (scale 0, zero codes), scale = -1 on some columns, a row
    with a large offset, and eps = 0."""
    M, K = 8, 512
    X, shift, scale, il = _adaln_inputs(181, M, K)
    X[0] = X[0, 5]
    X[1] = 0
    scale[:64] = 0xBF80                                        # -1
    Xf = bf16_to_f64(X).reshape(M, K).astype(np.float32)
    Xf[2] += 1000.0
    X = synth.to_bf16_bits(Xf)
    _check_adaln(X, shift, scale, il, M, K)
    _check_adaln(X, np.zeros(K, np.uint16), scale, il, M, K)
    _check_adaln(X, shift, scale, il, M, K, eps=0.0)


@pytest.mark.parametrize("M,N,K", [(300, 520, 1088), (2000, 4096, 4096)])
def test_route_modulated_against_the_oracle(M, N, K):
    """layer.route_modulated (adaLN step + W8A8 GEMM) against the oracle's
    modulation, quantization, int32 product and epilogue; protected layers
    are refused."""
    from paper_2606_12280_amd import layer
    X, shift, scale, _ = _adaln_inputs([184, M, N, K], M, K)
    rng = np.random.default_rng([185, M, N, K])
    W = synth.to_bf16_bits(rng.normal(0, 0.02, (N, K)).astype(np.float32))
    b = synth.to_bf16_bits(rng.normal(0, 0.01, N).astype(np.float32))
    lam = rng.uniform(0.25, 4.0, K).astype(np.float32)
    Wq_ref, ws_ref, il_ref = oracle.prepare_weight(W, lam, N, K)
    Xq_ref, xs_ref = oracle.adaln_quant_act(X, shift, scale, il_ref, M, K)
    acc = oracle.gemm_i32(Xq_ref, Wq_ref, M, N, K)
    Y_ref = oracle.epilogue(acc, xs_ref, ws_ref, b, M, N)
    Wd, bd = dev_bf16(W.reshape(N, K)), dev_bf16(b)
    lin = layer.prepare_linear(Wd, bd, dev(lam), protected=False)
    Y = layer.route_modulated(lin, dev_bf16(X.reshape(M, K)), dev_bf16(shift), dev_bf16(scale),
                              ws=layer.Workspace("cuda"))
    check_w8a8_output(host_bits(Y), Y_ref, acc, xs_ref, ws_ref, b)
    prot = layer.prepare_linear(Wd, bd, None, protected=True)
    with pytest.raises(ValueError):
        layer.route_modulated(prot, dev_bf16(X.reshape(M, K)), dev_bf16(shift), dev_bf16(scale))


def test_adaln_quant_act_full_size():
    """The FFN-up / QKV input of a DiT block, 4608 x 4096, whole tensor."""
    M, K = 4608, 4096
    _check_adaln(*_adaln_inputs(182, M, K), M, K)


# --------------------------------------------------------------------------
# GGUF linears without a bias, with one token, and through the router
# --------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", ["q8_0", "q4_k"])
@pytest.mark.parametrize("M,N", [(1, 65), (3, 1)])
def test_gguf_linear_without_bias_small(fmt, M, N):
    K = 512
    c = synth.linear_case([190, M, N, K], M, N, K)
    W = dev_bf16(c["W"].reshape(N, K))
    X = c["X"].reshape(M, K)
    if fmt == "q8_0":
        qs_ref, d_ref = oracle.q8_0_quantize(c["W"], N, K)
        Wd = oracle.q8_0_dequantize(qs_ref, d_ref, N, K)
        qs, d = ops.q8_0_quantize(W)
        Y = host_bits(ops.q8_0_linear(dev_bf16(X), qs, d, None))
    else:
        ref = oracle.q4_k_quantize(c["W"], N, K)
        Wd = oracle.q4_k_dequantize(ref, N, K)
        Y = host_bits(ops.q4_k_linear(dev_bf16(X), ops.q4_k_quantize(W), None))
    check_bf16_output(Y, X, Wd, None)


def test_router_runs_gguf_layers_like_the_entry_points():
    """layer.route on Q8_0 and Q4_K layers (decode into the shared workspace,
    then the bf16 linear) gives the entry points' outputs bit for bit."""
    from paper_2606_12280_amd import layer
    M, N, K = 96, 320, 768
    c = synth.linear_case([191, M, N, K], M, N, K, act="gelu")
    X, W, b = dev_bf16(c["X"].reshape(M, K)), dev_bf16(c["W"].reshape(N, K)), dev_bf16(c["bias"])
    ws = layer.Workspace(DEV)
    l8 = layer.prepare_q8_0(W, b)
    l4 = layer.prepare_q4_k(W, b)
    assert l8.weight_only and l4.weight_only and not l8.protected
    assert l4.nbytes() < l8.nbytes() < 2 * N * K
    y8 = host_bits(layer.route(l8, X, ws=ws))
    y4 = host_bits(layer.route(l4, X, ws=ws))
    assert np.array_equal(y8, host_bits(ops.q8_0_linear(X, l8.q8_qs, l8.q8_d, b)))
    assert np.array_equal(y4, host_bits(ops.q4_k_linear(X, l4.q4k, b)))


def test_empty_token_batch():
    """M = 0 (an empty batch, as a view with a live pointer and as a fresh
    tensor with a NULL one) through every entry point that takes tokens and
    through the router: [0, N] outputs, the running absmax unchanged, and the
    next full call bit-identical to the same call made before."""
    from paper_2606_12280_amd import layer
    M, N, K = 64, 320, 512
    c = synth.linear_case([197, M, N, K], M, N, K)
    X, W, b = dev_bf16(c["X"].reshape(M, K)), dev_bf16(c["W"].reshape(N, K)), dev_bf16(c["bias"])
    s = torch.zeros(K, dtype=torch.float32, device=DEV)
    ops.w8a8_act_absmax(X, s)
    lam = ops.w8a8_smooth_factors(s, W, 0.5)
    lays = [layer.prepare_linear(W, b, lam, protected=False),
            layer.prepare_linear(W, b, None, protected=True),
            layer.prepare_q8_0(W, b), layer.prepare_q4_k(W, b)]
    ws = layer.Workspace(DEV)
    before = [host_bits(layer.route(lay, X, ws=ws)) for lay in lays]
    shift = dev_bf16(synth.rand_bf16([198, 0], (K,), 0.05))
    scale = dev_bf16(synth.rand_bf16([198, 1], (K,), 0.1))
    ada_before = [host(t) for t in ops.w8a8_adaln_quant_act(X, shift, scale, lays[0].inv_lambda)]
    s_before = host(s)
    for X0 in (X[:0], torch.empty((0, K), dtype=torch.bfloat16, device=DEV)):
        ops.w8a8_act_absmax(X0, s)
        Xq0, xs0 = ops.w8a8_quant_act(X0, lays[0].inv_lambda)
        assert tuple(Xq0.shape) == (0, K) and tuple(xs0.shape) == (0,)
        assert tuple(ops.w8a8_linear(Xq0, xs0, lays[0].Wq, lays[0].w_scale, b).shape) == (0, N)
        assert tuple(ops.w8a8_gemm_i32(Xq0, lays[0].Wq).shape) == (0, N)
        assert tuple(ops.w8a8_adaln_quant_act(X0, shift, scale, lays[0].inv_lambda)[0].shape) == (0, K)
        for lay in lays:
            assert tuple(layer.route(lay, X0, ws=ws).shape) == (0, N)
            assert tuple(layer.route(lay, X0).shape) == (0, N)
    torch.cuda.synchronize()
    assert np.array_equal(host(s), s_before)
    for lay, y in zip(lays, before):
        assert np.array_equal(host_bits(layer.route(lay, X, ws=ws)), y)
    ada_after = [host(t) for t in ops.w8a8_adaln_quant_act(X, shift, scale, lays[0].inv_lambda)]
    assert all(np.array_equal(a, b_) for a, b_ in zip(ada_after, ada_before))


def test_binding_rejects_wrong_length_vectors():
    """Every 1-D operand must have exactly the length its matrix implies (the
    C ABI takes none, so a short vector would be read past its end): the
    binding raises ValueError before any launch and the preallocated outputs
    keep their contents."""
    M, N, K = 40, 96, 256
    c = synth.linear_case([199, M, N, K], M, N, K)
    X, W, b = dev_bf16(c["X"].reshape(M, K)), dev_bf16(c["W"].reshape(N, K)), dev_bf16(c["bias"])
    lam = torch.ones(K, dtype=torch.float32, device=DEV)
    Wq, ws, il = ops.w8a8_prepare_weight(W, lam)
    Xq, xs = ops.w8a8_quant_act(X, il)
    torch.cuda.synchronize()
    Y = torch.full((M, N), 7.0, dtype=torch.bfloat16, device=DEV)
    Xq_o = torch.full((M, K), 5, dtype=torch.int8, device=DEV)
    xs_o = torch.full((M,), 3.0, dtype=torch.float32, device=DEV)
    sh = dev_bf16(synth.rand_bf16([199, 0], (K,), 0.05))
    sc = dev_bf16(synth.rand_bf16([199, 1], (K,), 0.1))
    short = lambda t: t[:-1]
    long_ = lambda t: torch.cat([t, t[:1]])
    calls = [
        lambda f: ops.w8a8_linear(Xq, f(xs), Wq, ws, b, out=Y),
        lambda f: ops.w8a8_linear(Xq, xs, Wq, f(ws), b, out=Y),
        lambda f: ops.w8a8_linear(Xq, xs, Wq, ws, f(b), out=Y),
        lambda f: ops.bf16_linear(X, W, f(b), out=Y),
        lambda f: ops.w8a8_quant_act(X, f(il), Xq=Xq_o, x_scale=xs_o),
        lambda f: ops.w8a8_adaln_quant_act(X, f(sh), sc, il, Xq=Xq_o, x_scale=xs_o),
        lambda f: ops.w8a8_adaln_quant_act(X, sh, f(sc), il, Xq=Xq_o, x_scale=xs_o),
        lambda f: ops.w8a8_adaln_quant_act(X, sh, sc, f(il), Xq=Xq_o, x_scale=xs_o),
        lambda f: ops.w8a8_prepare_weight(W, f(lam)),
        lambda f: ops.w8a8_smooth_factors(f(lam), W),
        lambda f: ops.w8a8_act_absmax(X, f(lam.clone())),
    ]
    for call in calls:
        for f in (short, long_):
            with pytest.raises(ValueError, match="entries"):
                call(f)
    qs, d = ops.q8_0_quantize(W)
    with pytest.raises(ValueError, match="entries"):
        ops.q8_0_linear(X, qs, d, short(b), out=Y)
    with pytest.raises(ValueError, match="entries"):
        ops.q4_k_linear(X, ops.q4_k_quantize(W), short(b), out=Y)
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all()) and bool((Xq_o == 5).all()) and bool((xs_o == 3.0).all())


# --------------------------------------------------------------------------
# A seeded sweep of shapes: every tile configuration the dispatcher can pick
# (by round fill and by K % 128), ragged M and N, K from 64 to 4160 bytes.
# --------------------------------------------------------------------------

def _sweep_shapes(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        M = int(rng.choice([rng.integers(1, 65), rng.integers(65, 700), rng.integers(2000, 4700)]))
        N = int(rng.choice([rng.integers(1, 65), rng.integers(65, 1200), rng.integers(4000, 13000)]))
        K = 64 * int(rng.integers(1, 66))
        if M * N * K > 6e9:                     # keep the oracle's share to seconds
            K = 64 * max(1, int(6e9 / (M * N * 64)))
        out.append((M, N, K))
    return out


@pytest.mark.parametrize("M,N,K", _sweep_shapes(24, 195))
def test_w8a8_linear_shape_sweep(M, N, K):
    """int32 accumulators bit-exact, and the bf16 output within the
    epilogue's tolerance, on the shapes of a seeded sweep."""
    A = synth.rand_i8([196, M, K], (M, K))
    B = synth.rand_i8([197, N, K], (N, K))
    ref = oracle.gemm_i32(A, B, M, N, K)
    Ad, Bd = dev(A), dev(B)
    assert np.array_equal(host(ops.w8a8_gemm_i32(Ad, Bd)), ref)
    rng = np.random.default_rng([198, M, N, K])
    xs = rng.uniform(1e-3, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-4, 1e-2, N).astype(np.float32)
    b = synth.rand_bf16([199, N], (N,), 0.5)
    Y = host_bits(ops.w8a8_linear(Ad, dev(xs), Bd, dev(ws), dev_bf16(b)))
    check_w8a8_output(Y, oracle.epilogue(ref, xs, ws, b, M, N), ref, xs, ws, b)


def _quant_sweep(n, seed):
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, 3000)), 64 * int(rng.integers(1, 257))) for _ in range(n)]


@pytest.mark.parametrize("M,K", _quant_sweep(16, 200))
def test_quant_act_shape_sweep(M, K):
    """Codes and scales bit-exact on a seeded sweep of (M, K), every row-group
    configuration of the quant kernel up to K = 16384."""
    c = synth.linear_case([201, M, K], M, 8, K, act="outlier")
    lam = np.random.default_rng([202, K]).uniform(0.25, 4.0, K).astype(np.float32)
    Xq, xs, Xq_ref, xs_ref = _quant_case(c["X"], lam, M, K)
    assert np.array_equal(xs.view(np.uint32), xs_ref.view(np.uint32))
    assert np.array_equal(Xq, Xq_ref)


@pytest.mark.parametrize("M,N,K", _sweep_shapes(10, 203))
def test_bf16_linear_shape_sweep(M, N, K):
    c = synth.linear_case([204, M, N, K], M, N, K)
    Y = host_bits(ops.bf16_linear(dev_bf16(c["X"]), dev_bf16(c["W"]), dev_bf16(c["bias"])))
    rows = np.random.default_rng([205, M]).choice(M, min(M, 64), replace=False)
    check_bf16_output(Y[rows], c["X"].reshape(M, K)[rows], c["W"].reshape(N, K), c["bias"])
