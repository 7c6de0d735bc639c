"""Pins of the CPU oracle against facts fixed outside it (CPU only).

Each test checks the oracle against something other than itself: a library
routine computing a textbook special case, a closed-form bound, an invariant,
or brute force on tiny inputs. The recipe is the paper's Section 3 ("INT8
W8A8"): per-output-row INT8 weights, per-token dynamic INT8 activations,
SmoothQuant smoothing with lambda_j = s_j^alpha / max_i |W_ij|^(1-alpha), and
bf16 protection of fragile layers. Each test names the mistake it would catch.
"""
from __future__ import annotations

import hashlib
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from bf16ref import bf16_to_f64, round_bf16_exact, ulp_distance

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
QUANT_SLACK = 0.5 + 2.0 ** -14   # |q*s - x'| <= s*(1/2 + fp32 slack)


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build()


# --------------------------------------------------------------------------
# bf16 conversions
# --------------------------------------------------------------------------

def test_bf16_widening_matches_bit_layout():
    bits = np.array([0x0000, 0x8000, 0x3F80, 0xBF80, 0x4300, 0x0001, 0x7F7F, 0x3E80],
                    np.uint16)
    want = [0.0, -0.0, 1.0, -1.0, 128.0, 2.0 ** -133, float(bf16_to_f64([0x7F7F])[0]), 0.25]
    got = [oracle.bf16_to_float(int(b)) for b in bits]
    assert got == want


def test_double_to_bf16_matches_exact_rounding():
    """Ties-to-even, subnormals and overflow against brute-force rational
    rounding (catches round-half-up, double rounding through binary32,
    wrong subnormal spacing)."""
    rng = np.random.default_rng(11)
    vals = list(rng.standard_normal(300) * 10.0 ** rng.integers(-40, 38, 300))
    # exact ties: midpoints between neighbouring bf16 values
    for h in (0x3F80, 0x3F81, 0x4000, 0x0001, 0x0002, 0x7F7E, 0x4B00):
        lo = Fraction(float(bf16_to_f64([h])[0]))
        hi = Fraction(float(bf16_to_f64([h + 1])[0]))
        mid = (lo + hi) / 2
        vals += [float(mid), -float(mid)]
    # a value that double-rounds wrongly through binary32: 1 + 2^-8 + 2^-30
    vals += [1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -8 - 2.0 ** -30]
    vals += [3.0e38, 3.3961e38, -3.4e38, 1e-45, 2.0 ** -134, 2.0 ** -134 * 3]
    for v in vals:
        assert oracle.double_to_bf16(v) == round_bf16_exact(v), v


# --------------------------------------------------------------------------
# the int32 product
# --------------------------------------------------------------------------

@pytest.mark.parametrize("M,N,K,seed", [(1, 1, 64, 0), (3, 5, 64, 1), (17, 9, 128, 2),
                                        (65, 33, 256, 3), (2, 64, 1024, 4)])
def test_gemm_i32_matches_numpy_int64(M, N, K, seed):
    """Brute force against NumPy's int64 matmul (catches transposed operands,
    dropped terms, sign-extension mistakes)."""
    A = synth.rand_i8([seed, 0], (M, K))
    B = synth.rand_i8([seed, 1], (N, K))
    ref = A.astype(np.int64) @ B.astype(np.int64).T
    got = oracle.gemm_i32(A, B, M, N, K)
    assert np.array_equal(got.astype(np.int64), ref)


def test_gemm_i32_extreme_magnitudes():
    """All +-127 operands at K = 16384 reach 127^2 K = 2.64e8 without overflow."""
    K = 16384
    A = np.full((2, K), 127, np.int8)
    A[1] = -127
    B = np.full((3, K), -127, np.int8)
    B[2, ::2] = 127
    got = oracle.gemm_i32(A, B, 2, 3, K)
    ref = A.astype(np.int64) @ B.astype(np.int64).T
    assert np.array_equal(got, ref)
    assert abs(int(got[0, 0])) == 127 * 127 * K


# --------------------------------------------------------------------------
# calibration and the smoothing factor
# --------------------------------------------------------------------------

def test_act_absmax_matches_numpy_and_accumulates():
    X = synth.rand_bf16(5, (37, 96), 3.0)
    got = oracle.act_absmax(X, 37, 96)
    assert np.array_equal(got, np.abs(bf16_to_f64(X)).max(0).astype(np.float32))
    X2 = synth.rand_bf16(6, (5, 96), 9.0)
    got2 = oracle.act_absmax(X2, 5, 96, got)
    ref2 = np.maximum(got, np.abs(bf16_to_f64(X2)).max(0).astype(np.float32))
    assert np.array_equal(got2, ref2)


def _bf16_col(vals):
    return synth.to_bf16_bits(np.array(vals, np.float32))


def test_smooth_factors_closed_forms():
    """lambda = s^a / m^(1-a) on powers of two (catches a swapped exponent,
    s and m swapped, or max over the wrong axis of W)."""
    # K = 4 input channels, N = 2 output rows; column maxima m = [1, 4, 2, 3]
    W = np.stack([_bf16_col([1.0, -4.0, 0.5, 0.0]), _bf16_col([-0.25, 2.0, -2.0, 3.0])])
    s = np.array([4.0, 1.0, 2.0, 0.0], np.float32)   # last channel: s = 0
    lam = oracle.smooth_factors(s, W, 2, 4, 0.5)
    assert lam.tolist() == [2.0, 0.5, 1.0, 1.0]
    lam3 = oracle.smooth_factors(np.array([8.0, 1, 1, 1], np.float32), W, 2, 4, 1.0 / 3.0)
    # 8^(1/3) / 1^(2/3) = 2
    assert abs(float(lam3[0]) - 2.0) <= 2.0 * 2.0 ** -23
    # 1^(1/3) / 4^(2/3) = 2^(-4/3)
    assert abs(float(lam3[1]) - 2.0 ** (-4.0 / 3.0)) <= 2.0 ** -23


@pytest.mark.parametrize("alpha", [0.5, 0.25, 0.8])
def test_smoothing_balances_channel_ranges(alpha):
    """SmoothQuant's purpose: after X/lambda and W*lambda the per-channel
    ranges obey (s/lambda) / (m*lambda) = (s m)^(1 - 2 alpha); at alpha = 0.5
    activation and weight channels end up with equal absmax."""
    c = synth.tiny_case()
    M, N, K = c["M"], c["N"], c["K"]
    s = oracle.act_absmax(c["X"], M, K)
    lam = oracle.smooth_factors(s, c["W"], N, K, alpha).astype(np.float64)
    x_rng = np.abs(bf16_to_f64(c["X"]).reshape(M, K)).max(0) / lam
    w_rng = np.abs(bf16_to_f64(c["W"]).reshape(N, K)).max(0) * lam
    lhs = np.log(x_rng / w_rng)
    rhs = (1.0 - 2.0 * alpha) * np.log(x_rng * lam * w_rng / lam)
    assert np.allclose(lhs, rhs, atol=1e-6)


def test_inv_lambda_is_correctly_rounded_reciprocal():
    """inv_lambda = RN32(1/lambda): double rounding of a binary64 quotient to
    binary32 is innocuous (53 >= 2*24 + 2), so NumPy gives the exact answer.
    Also pins the SmoothQuant identity (X diag(1/l))(diag(l) W^T) = X W^T."""
    rng = np.random.default_rng(3)
    lam = np.exp(rng.uniform(-6, 6, 512)).astype(np.float32)
    W = synth.rand_bf16(4, (8, 512), 0.02)
    _, _, il = oracle.prepare_weight(W, lam, 8, 512)
    want = (1.0 / lam.astype(np.float64)).astype(np.float32)
    assert np.array_equal(il, want)
    X = bf16_to_f64(synth.rand_bf16(5, (16, 512))).reshape(16, 512)
    Wf = bf16_to_f64(W).reshape(8, 512)
    lhs = (X * il.astype(np.float64)) @ (Wf * lam.astype(np.float64)).T
    ref = X @ Wf.T
    assert np.linalg.norm(lhs - ref) <= 2.0 ** -22 * np.linalg.norm(np.abs(X) @ np.abs(Wf).T)


# --------------------------------------------------------------------------
# per-row quantization
# --------------------------------------------------------------------------

def test_round_half_even_ties():
    """With lambda = 1 and a row whose absmax is 127, scale = 1 and the codes
    are rint(x): NumPy's rint (ties to even) fixes them. Catches round-half-up
    or round-half-away-from-zero."""
    row = np.array([127.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5, 126.5, -126.5,
                    0.25, 0.75, -0.75, 64.5, 65.5, 0.0], np.float32)
    K = 64
    x = np.zeros(K, np.float32)
    x[: row.size] = row
    X = synth.to_bf16_bits(x)[None, :]
    ones = np.ones(K, np.float32)
    Xq, xs = oracle.quant_act(X, ones, 1, K)
    assert xs[0] == np.float32(1.0)
    assert np.array_equal(Xq[0].astype(np.float64), np.rint(x.astype(np.float64)))


def _dequant_bound_ok(q, s, exact):
    err = np.abs(q.astype(np.float64) * s.astype(np.float64)[:, None] - exact)
    return np.all(err <= s.astype(np.float64)[:, None] * QUANT_SLACK)


def test_activation_quant_invariants_tiny():
    """max|q| = 127 on every nonzero row and |q s - X/lambda| <= s/2 (plus
    binary32 slack) against X/lambda in binary64 (catches multiplying by
    lambda instead of dividing, a wrong scale or a per-tensor scale)."""
    c = synth.tiny_case()
    M, N, K = c["M"], c["N"], c["K"]
    r = oracle.recipe(c["X"], c["W"], c["bias"], M, N, K)
    Xq, xs = r["Xq"], r["x_scale"]
    assert np.all(np.abs(Xq.astype(np.int32)).max(1) == 127)
    assert Xq.min() >= -127
    exact = bf16_to_f64(c["X"]).reshape(M, K) / r["lambda"].astype(np.float64)
    assert _dequant_bound_ok(Xq, xs, exact)
    # the scale is absmax/127 of the smoothed row, correctly rounded
    amax = np.abs((bf16_to_f64(c["X"]).reshape(M, K).astype(np.float32)
                   * r["inv_lambda"][None, :]).astype(np.float32)).max(1)
    assert np.array_equal(xs, (amax.astype(np.float64) / 127.0).astype(np.float32))


def test_weight_quant_invariants_tiny():
    """Same for the per-output-row weight codes against W*lambda."""
    c = synth.tiny_case()
    M, N, K = c["M"], c["N"], c["K"]
    r = oracle.recipe(c["X"], c["W"], c["bias"], M, N, K)
    Wq, ws = r["Wq"], r["w_scale"]
    assert np.all(np.abs(Wq.astype(np.int32)).max(1) == 127)
    exact = bf16_to_f64(c["W"]).reshape(N, K) * r["lambda"].astype(np.float64)
    assert _dequant_bound_ok(Wq, ws, exact)


def test_quant_special_rows():
    """Zero row -> scale 0, codes 0; constant row -> all +-127; a row below
    2^-96 -> zero (reciprocal would overflow); one nonzero entry -> +-127."""
    K = 128
    rows = np.zeros((5, K), np.float32)
    rows[1, :] = -3.0
    rows[2, :] = 2.0 ** -100
    rows[3, 17] = 0.375
    rows[4, :] = 1.0
    rows[4, ::3] = -1.0
    X = synth.to_bf16_bits(rows)
    Xq, xs = oracle.quant_act(X, np.ones(K, np.float32), 5, K)
    assert xs[0] == 0 and not Xq[0].any()
    assert np.all(Xq[1] == -127) and xs[1] == np.float32(3.0 / 127.0)
    assert xs[2] == 0 and not Xq[2].any()
    assert Xq[3, 17] == 127 and np.count_nonzero(Xq[3]) == 1
    assert np.array_equal(np.abs(Xq[4]), np.full(K, 127, np.int8))
    assert np.all(Xq[4, ::3] == -127)


# --------------------------------------------------------------------------
# the whole recipe
# --------------------------------------------------------------------------

def _grid_case(rng, M, N, K):
    """Inputs on the INT8 grid: X_tk = a_t i_tk lambda_k, W_nk = c_n j_nk /
    lambda_k with powers of two a, c, lambda and integer i, j in [-127, 127],
    every row holding a +-127. Quantization is then lossless, so the recipe
    must return bf16(X W^T + b) exactly."""
    lam = (2.0 ** rng.integers(-2, 3, K)).astype(np.float32)
    a = 2.0 ** rng.integers(-6, 2, M)
    cw = 2.0 ** rng.integers(-9, -4, N)
    i = rng.integers(-127, 128, (M, K))
    j = rng.integers(-127, 128, (N, K))
    i[np.arange(M), rng.integers(0, K, M)] = 127
    j[np.arange(N), rng.integers(0, K, N)] = -127
    X = a[:, None] * i * lam[None, :]
    W = cw[:, None] * j / lam[None, :]
    b = rng.integers(-64, 64, N) * 2.0 ** -8
    bits = lambda v: synth.to_bf16_bits(np.asarray(v, np.float32))
    return bits(X), bits(W), bits(b), lam, X, W, b


def test_lossless_grid_reduces_to_plain_product():
    """Special case reducing to an exact matmul: catches the smoothing
    direction, transposes, scale mistakes and a dropped bias exactly."""
    rng = np.random.default_rng(21)
    M, N, K = 9, 7, 128
    Xb, Wb, bb, lam, X, W, b = _grid_case(rng, M, N, K)
    assert np.array_equal(bf16_to_f64(Xb).reshape(M, K), X)   # grid is bf16-exact
    assert np.array_equal(bf16_to_f64(Wb).reshape(N, K), W)
    r = oracle.recipe(Xb, Wb, bb, M, N, K, lam=lam)
    exact = X @ W.T + b[None, :]          # every term is a small dyadic: exact
    want = np.array([[round_bf16_exact(float(v)) for v in row] for row in exact],
                    np.uint16)
    assert np.array_equal(r["Y"], want)
    assert np.array_equal(r["acc"].astype(np.float64) * r["x_scale"][:, None]
                          * r["w_scale"][None, :], X @ W.T)
    # the fused per-row routine (the one the CPU baseline times) on the same
    # lossless grid, with and without the bias
    Yf = oracle.w8a8_linear(r["Xq"], r["x_scale"], r["Wq"], r["w_scale"], bb, M, N, K)
    assert np.array_equal(Yf, want)
    Y0 = oracle.w8a8_linear(r["Xq"], r["x_scale"], r["Wq"], r["w_scale"], None, M, N, K)
    want0 = np.array([[round_bf16_exact(float(v)) for v in row] for row in X @ W.T], np.uint16)
    assert np.array_equal(Y0, want0)


@pytest.mark.parametrize("which", ["tiny", "gelu_small"])
def test_w8a8_error_bound_vs_fp64(which):
    """Closed-form W8A8 error bound against binary64 X W^T + b, elementwise:
    with x' = q_x s_x + e_x, w' = q_w s_w + e_w and |e| <= c s,
    |acc s_x s_w - sum x w| <= c s_w sum|q_x s_x| + c s_x sum|q_w s_w| + K c^2 s_x s_w,
    plus the final bf16 rounding (half an ulp)."""
    if which == "tiny":
        c = synth.tiny_case()
    else:
        c = synth.linear_case([77], 48, 80, 512, act="gelu")
    M, N, K = c["M"], c["N"], c["K"]
    r = oracle.recipe(c["X"], c["W"], c["bias"], M, N, K)
    X = bf16_to_f64(c["X"]).reshape(M, K)
    W = bf16_to_f64(c["W"]).reshape(N, K)
    b = bf16_to_f64(c["bias"])
    ref = X @ W.T + b[None, :]
    sx = r["x_scale"].astype(np.float64)[:, None]
    sw = r["w_scale"].astype(np.float64)[None, :]
    dqx = np.abs(r["Xq"].astype(np.float64)) * sx
    dqw = np.abs(r["Wq"].astype(np.float64)) * sw.T
    cc = QUANT_SLACK
    bound = cc * sw * dqx.sum(1)[:, None] + cc * sx * dqw.sum(1)[None, :] + K * cc * cc * sx * sw
    y = bf16_to_f64(r["Y"]).reshape(M, N)
    total = bound + 2.0 ** -8 * np.abs(y) + 1e-30
    assert np.all(np.abs(y - ref) <= total)
    # and the bound is not vacuous: the relative error is small overall
    assert np.linalg.norm(y - ref) <= 0.05 * np.linalg.norm(ref)


def test_epilogue_against_exact_rationals():
    """bf16(acc * s_x * s_w + b) against exact rational arithmetic with the
    brute-force rounding (catches a dropped bias, a wrong scale index or
    rounding through binary32)."""
    rng = np.random.default_rng(8)
    M, N = 6, 40
    C = rng.integers(-2 ** 28, 2 ** 28, (M, N), dtype=np.int64).astype(np.int32)
    xs = rng.uniform(1e-4, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-5, 1e-2, N).astype(np.float32)
    b = synth.rand_bf16(9, (N,), 50.0)
    Y = oracle.epilogue(C, xs, ws, b, M, N)
    bf = bf16_to_f64(b)
    for t in range(M):
        for n in range(N):
            exact = (Fraction(int(C[t, n])) * Fraction(float(xs[t])) * Fraction(float(ws[n]))
                     + Fraction(float(bf[n])))
            assert Y[t, n] == round_bf16_exact(exact), (t, n)
    Y0 = oracle.epilogue(C, xs, ws, None, M, N)
    assert Y0[2, 3] == round_bf16_exact(Fraction(int(C[2, 3])) * Fraction(float(xs[2]))
                                        * Fraction(float(ws[3])))


def test_w8a8_linear_against_int64_and_exact_rationals():
    """The fused routine (int32 sum and epilogue per row, what the CPU
    baseline times) against an int64 NumPy product and exact rational
    epilogue arithmetic, on a ragged shape with codes reaching +-127 (catches
    a dropped last k, a dropped bias, a wrong scale index or a transposed
    operand)."""
    rng = np.random.default_rng(31)
    M, N, K = 7, 33, 320
    Xq = rng.integers(-127, 128, (M, K)).astype(np.int8)
    Wq = rng.integers(-127, 128, (N, K)).astype(np.int8)
    Xq[:, -1] = 127                      # the last k carries weight in every sum
    Wq[:, -1] = -127
    C = Xq.astype(np.int64) @ Wq.astype(np.int64).T
    xs = rng.uniform(1e-4, 1e-1, M).astype(np.float32)
    ws = rng.uniform(1e-5, 1e-2, N).astype(np.float32)
    b = synth.rand_bf16(10, (N,), 5.0)
    bf = bf16_to_f64(b)
    Y = oracle.w8a8_linear(Xq, xs, Wq, ws, b, M, N, K)
    Y0 = oracle.w8a8_linear(Xq, xs, Wq, ws, None, M, N, K)
    for t in range(M):
        for n in range(N):
            p = Fraction(int(C[t, n])) * Fraction(float(xs[t])) * Fraction(float(ws[n]))
            assert Y[t, n] == round_bf16_exact(p + Fraction(float(bf[n]))), (t, n)
            assert Y0[t, n] == round_bf16_exact(p), (t, n)


def test_bf16_linear_small_integers_exact():
    """Protected path on small integers: every partial sum is exact, so the
    result is bf16 of the integer product (brute-force rounding)."""
    rng = np.random.default_rng(2)
    M, N, K = 5, 6, 200
    X = rng.integers(-8, 9, (M, K)).astype(np.float64)
    W = rng.integers(-8, 9, (N, K)).astype(np.float64)
    b = rng.integers(-100, 100, N).astype(np.float64)
    Y = oracle.bf16_linear(synth.to_bf16_bits(X), synth.to_bf16_bits(W),
                           synth.to_bf16_bits(b), M, N, K)
    exact = X @ W.T + b
    want = np.array([[round_bf16_exact(float(v)) for v in row] for row in exact], np.uint16)
    assert np.array_equal(Y, want)


def test_bf16_linear_random_vs_numpy_fp64():
    """Random bf16 inputs against BLAS binary64 plus exact rounding: equal up
    to a binary64 summation-order difference at a bf16 rounding boundary."""
    M, N, K = 8, 16, 512
    X = synth.rand_bf16(31, (M, K))
    W = synth.rand_bf16(32, (N, K), 0.05)
    b = synth.rand_bf16(33, (N,), 0.1)
    Y = oracle.bf16_linear(X, W, b, M, N, K)
    ref = bf16_to_f64(X).reshape(M, K) @ bf16_to_f64(W).reshape(N, K).T + bf16_to_f64(b)
    want = np.array([[round_bf16_exact(float(v)) for v in row] for row in ref], np.uint16)
    d = ulp_distance(Y, want)
    assert d.max() <= 1 and (d == 0).mean() > 0.99


def test_oracle_thread_count_invariance():
    c = synth.linear_case([12], 33, 40, 256)
    r1 = oracle.recipe(c["X"], c["W"], c["bias"], 33, 40, 256)
    n = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        r2 = oracle.recipe(c["X"], c["W"], c["bias"], 33, 40, 256)
    finally:
        oracle.set_num_threads(n)
    for key in r1:
        assert np.array_equal(r1[key], r2[key]), key


def _digest(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def test_tiny_case_digest_is_stable():
    """Inputs and oracle outputs of the tiny case against the digests stored
    by tests/golden/make_golden.py (catches a drifting RNG stream or an
    unintended change to the oracle's arithmetic)."""
    with open(os.path.join(GOLDEN, "tiny_case_digest.json")) as f:
        want = json.load(f)
    c = synth.tiny_case()
    r = oracle.recipe(c["X"], c["W"], c["bias"], c["M"], c["N"], c["K"])
    got = {"X": _digest(c["X"]), "W": _digest(c["W"]), "bias": _digest(c["bias"])}
    got.update({k: _digest(v) for k, v in r.items()})
    assert got == want["sha256"]


# --------------------------------------------------------------------------
# fragility profile (Section 3, "Activation-fragility profiling and
# protection"): max |x|, standard deviation, kurtosis; top-N; Spearman
# --------------------------------------------------------------------------

def _exact_moments(vals):
    """max |x|, mean, m2, m4 of bf16 values as exact rationals."""
    fr = [Fraction(float(v)) for v in vals]
    n = len(fr)
    mean = sum(fr) / n
    m2 = sum((x - mean) ** 2 for x in fr) / n
    m4 = sum((x - mean) ** 4 for x in fr) / n
    return max(abs(x) for x in fr), mean, m2, m4


def test_act_moments_against_exact_rationals():
    """Catches a missing centering, a sample (n-1) variance, an excess
    (minus 3) kurtosis, a signed maximum or a dropped row."""
    for seed, (M, K) in enumerate([(3, 7), (5, 16), (1, 33)]):
        X = synth.rand_bf16([120, seed], (M, K), 1.0)
        X[0, 0] = synth.to_bf16_bits(np.array([-5.25], np.float32))[0]  # largest magnitude, negative
        X[-1, -1] = synth.to_bf16_bits(np.array([4.5], np.float32))[0]
        got = oracle.act_moments(X, M, K)
        amax, mean, m2, m4 = _exact_moments(bf16_to_f64(X.ravel()))
        assert got[0] == float(amax) == 5.25
        assert abs(got[1] - float(mean)) <= 1e-15 * max(1.0, abs(float(mean)))
        assert got[2] == pytest.approx(float(m2) ** 0.5, rel=1e-14)
        assert got[3] == pytest.approx(float(m4 / (m2 * m2)), rel=1e-13)


def test_act_moments_two_point_and_constant():
    a = synth.to_bf16_bits(np.array([0.375, -0.375], np.float32))
    got = oracle.act_moments(np.tile(a, 12), 3, 8)
    assert list(got) == [0.375, 0.0, 0.375, 1.0]        # kurtosis of +-a is exactly 1
    c = np.full((4, 9), synth.to_bf16_bits(np.array([-2.5], np.float32))[0], np.uint16)
    assert list(oracle.act_moments(c, 4, 9)) == [2.5, -2.5, 0.0, 0.0]   # constant: kurtosis 0


def test_act_moments_textbook_kurtosis():
    """Sample kurtosis of large bf16 samples against the distributions'
    values: Gaussian 3, uniform 9/5, Laplace 6 (tolerances ~10 standard
    errors; bf16 rounding moves them by far less)."""
    rng = np.random.default_rng(121)
    n = 1 << 21
    cases = [(rng.standard_normal(n), 3.0, 0.035), (rng.uniform(-1, 1, n), 1.8, 0.01),
             (rng.laplace(0, 1, n), 6.0, 0.2)]
    for x, want, tol in cases:
        b = synth.to_bf16_bits(x.astype(np.float32)).reshape(1024, -1)
        got = oracle.act_moments(b, b.shape[0], b.shape[1])
        assert abs(got[3] - want) < tol, (want, got[3])


def test_act_moments_shift_and_scale():
    """Integer-valued inputs: adding 64 (exact in bf16) shifts the mean only;
    doubling scales max and std by 2 and leaves the kurtosis."""
    rng = np.random.default_rng(122)
    v = rng.integers(-60, 61, (37, 19)).astype(np.float32)
    base = oracle.act_moments(synth.to_bf16_bits(v), 37, 19)
    sh = oracle.act_moments(synth.to_bf16_bits(v + 64.0), 37, 19)
    dbl = oracle.act_moments(synth.to_bf16_bits(2.0 * v), 37, 19)
    assert sh[1] == pytest.approx(base[1] + 64.0, rel=1e-15)
    assert sh[2] == pytest.approx(base[2], rel=1e-12)
    assert sh[3] == pytest.approx(base[3], rel=1e-10)
    assert dbl[0] == 2 * base[0] and dbl[2] == pytest.approx(2 * base[2], rel=1e-15)
    assert dbl[3] == pytest.approx(base[3], rel=1e-14)


def test_act_moments_matches_scipy():
    from scipy import stats
    c = synth.linear_case([123], 64, 8, 512, act="gelu")
    x = bf16_to_f64(c["X"]).ravel()
    got = oracle.act_moments(c["X"], 64, 512)
    assert got[0] == np.abs(x).max()
    assert got[1] == pytest.approx(x.mean(), rel=1e-13)
    assert got[2] == pytest.approx(x.std(), rel=1e-13)
    assert got[3] == pytest.approx(stats.kurtosis(x, fisher=False, bias=True), rel=1e-11)


def test_act_moments_thread_invariant():
    c = synth.linear_case([124], 77, 8, 320, act="gelu")
    a = oracle.act_moments(c["X"], 77, 320)
    n = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        b = oracle.act_moments(c["X"], 77, 320)
    finally:
        oracle.set_num_threads(n)
    assert np.array_equal(a, b)


def test_fragility_scores_top_n_and_spearman():
    from scipy import stats
    k = np.array([[3.0, 5.0], [10.0, 12.0], [4.0, 4.0], [11.0, 11.0]])
    assert list(oracle.fragility_scores(k)) == [4.0, 11.0, 4.0, 11.0]
    assert oracle.top_n(oracle.fragility_scores(k), 3) == [1, 3, 0]   # ties by index
    rng = np.random.default_rng(125)
    for _ in range(20):
        s = rng.integers(0, 6, 30).astype(float)        # many ties
        n = int(rng.integers(0, 31))
        brute = sorted(range(30), key=lambda i: (-s[i], i))[:n]
        assert oracle.top_n(s, n) == brute
        a, b = rng.integers(0, 8, 25), rng.normal(size=25)
        assert oracle.spearman(a, b) == pytest.approx(stats.spearmanr(a, b).statistic, abs=1e-12)
    assert oracle.spearman([1, 2, 3], [10, 20, 30]) == pytest.approx(1.0)
    assert oracle.spearman([1, 2, 3], [3, 2, 1]) == pytest.approx(-1.0)


# --------------------------------------------------------------------------
# GGUF Q8_0 weight-only (Section 3, "GGUF k-quants": 8.5 bits per weight,
# round to nearest)
# --------------------------------------------------------------------------

def test_half_conversion_matches_numpy():
    """binary16 rounding (ties to even, subnormals, overflow) against numpy,
    and widening of every finite bit pattern."""
    rng = np.random.default_rng(140)
    vals = np.concatenate([rng.normal(0, 1, 2000), rng.normal(0, 1e-5, 2000),
                           rng.uniform(-70000, 70000, 2000), 2.0 ** rng.uniform(-26, -13, 2000),
                           [65504.0, 65519.9, 65520.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26,
                            2.0 ** -14 * (1 - 2.0 ** -11), 1 + 2.0 ** -11, 1 + 3 * 2.0 ** -11]]
                          ).astype(np.float32)
    with np.errstate(over="ignore"):
        want = vals.astype(np.float16).view(np.uint16)
    got = np.array([oracle.float_to_half(float(v)) for v in vals], np.uint16)
    assert np.array_equal(got, want)
    bits = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    finite = (bits & 0x7c00) != 0x7c00
    wide = np.array([oracle.half_to_float(int(b)) for b in bits[finite]], np.float32)
    assert np.array_equal(wide, bits[finite].view(np.float16).astype(np.float32))


def _f16(bits) -> np.ndarray:
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float32)


def test_q8_0_invariants():
    """Codes in [-127, 127], 127 reached in every block, scale = amax/127
    to binary16 precision, reconstruction within half a step."""
    N, K = 48, 256
    W = synth.rand_bf16([141], (N, K), 0.02)
    qs, d = oracle.q8_0_quantize(W, N, K)
    w = bf16_to_f64(W).reshape(N, K // 32, 32)
    q = qs.reshape(N, K // 32, 32).astype(np.float64)
    ds = _f16(d).astype(np.float64)[..., None]
    amax = np.abs(w).max(axis=2)
    assert np.abs(q).max() <= 127
    assert np.array_equal(np.abs(q).max(axis=2), np.full_like(amax, 127))
    assert np.allclose(ds[..., 0], amax / 127, rtol=2.0 ** -11)
    assert np.all(np.abs(w - ds * q) <= ds * (0.5 + 2.0 ** -12))


def test_q8_0_exact_grid_and_ties():
    """Multiples of 1/16 with a block maximum of 127/16: the scale is exact
    and every weight reads back exactly. With scale 1: +-0.5, 2.5, 3.5 tie
    to even."""
    rng = np.random.default_rng(142)
    k = rng.integers(-127, 128, (8, 64)).astype(np.float32)
    k[:, 0] = 127
    k[:, 32] = -127
    W = synth.to_bf16_bits(k / 16)
    qs, d = oracle.q8_0_quantize(W, 8, 64)
    assert np.all(_f16(d) == 1 / 16)
    assert np.array_equal(qs, k.astype(np.int8))
    assert np.array_equal(oracle.q8_0_dequantize(qs, d, 8, 64), W)
    t = np.array([127.0, 0.5, -0.5, 1.5, 2.5, -2.5, 3.5, 126.5] + [0.0] * 24, np.float32)
    qs, d = oracle.q8_0_quantize(synth.to_bf16_bits(t), 1, 32)
    assert _f16(d)[0, 0] == 1.0
    assert list(qs[0, :8]) == [127, 0, 0, 2, 2, -2, 4, 126]


def test_q8_0_special_blocks():
    """A zero block (scale 0, zero codes), a block whose scale underflows
    binary16 (zero codes), and a block whose scale is capped at 65504 (codes
    clamp at +-127)."""
    W = np.zeros((1, 96), np.float32)
    W[0, 32:64] = 2.0 ** -30
    W[0, 64] = 9.0e6
    W[0, 65] = -1.0e6
    B = synth.to_bf16_bits(W)
    qs, d = oracle.q8_0_quantize(B, 1, 96)
    assert d[0, 0] == 0 and not qs[0, :32].any()
    assert d[0, 1] == 0 and not qs[0, 32:64].any()
    assert _f16(d)[0, 2] == 65504.0
    assert qs[0, 64] == 127 and qs[0, 65] == round(-1.0e6 / 65504.0)


def test_q8_0_dequantize_is_one_rounding():
    rng = np.random.default_rng(143)
    qs = rng.integers(-127, 128, (5, 64)).astype(np.int8)
    d = np.array([[oracle.float_to_half(float(v)) for v in rng.lognormal(-6, 3, 2)] for _ in range(5)],
                 np.uint16)
    got = oracle.q8_0_dequantize(qs, d, 5, 64)
    for n in range(5):
        for kk in range(64):
            exact = Fraction(float(_f16(d[n, kk // 32]))) * int(qs[n, kk])
            assert got[n, kk] == round_bf16_exact(exact)


def test_q8_0_linear_against_numpy_fp64():
    """The weight-only linear against binary64 X W'^T + b on the decoded
    weights, within the binary32 summation bound plus one bf16 rounding."""
    c = synth.linear_case([144], 33, 40, 256)
    qs, d = oracle.q8_0_quantize(c["W"], 40, 256)
    Wd = oracle.q8_0_dequantize(qs, d, 40, 256)
    Y = oracle.q8_0_linear(c["X"], qs, d, c["bias"], 33, 40, 256)
    X = bf16_to_f64(c["X"]).reshape(33, 256)
    ref = X @ bf16_to_f64(Wd).reshape(40, 256).T + bf16_to_f64(c["bias"])[None, :]
    y = bf16_to_f64(Y).reshape(33, 40)
    assert np.all(np.abs(y - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-30)
    # and the quantization error of the weights stays within half a step
    Wf = bf16_to_f64(c["W"]).reshape(40, 8, 32)
    step = _f16(d).astype(np.float64)[..., None]
    assert np.all(np.abs(bf16_to_f64(Wd).reshape(40, 8, 32) - Wf) <= step * 0.5 + np.abs(Wf) * 2.0 ** -8)


# --------------------------------------------------------------------------
# GGUF Q4_K weight-only (Section 3, "GGUF k-quants": 4-bit codes in
# super-blocks of 256 weights, 8 sub-blocks of 32 with 6-bit scales and
# offsets under binary16 super-block scales)
# --------------------------------------------------------------------------

def _pack_k4(sc, mn):
    """Test-side packer of the 12-byte k-quant scale layout, written from its
    definition: for j < 4, byte j = sc_j and byte j + 4 = m_j (low 6 bits);
    for j >= 4, byte j + 4 = (sc_j & 15) | (m_j & 15) << 4, and the top two
    bits of sc_j and m_j go to the top of bytes j - 4 and j. sc, mn are
    [..., 8]; returns [..., 12]."""
    sc = np.asarray(sc, np.uint32)
    mn = np.asarray(mn, np.uint32)
    out = np.zeros(sc.shape[:-1] + (12,), np.uint32)
    out[..., 0:4] = (sc[..., 0:4] & 63) | ((sc[..., 4:8] >> 4) << 6)
    out[..., 4:8] = (mn[..., 0:4] & 63) | ((mn[..., 4:8] >> 4) << 6)
    out[..., 8:12] = (sc[..., 4:8] & 15) | ((mn[..., 4:8] & 15) << 4)
    return out.astype(np.uint8)


def _unpack_k4(packed):
    """Inverse of _pack_k4: [..., 12] -> (sc [..., 8], mn [..., 8])."""
    b = np.asarray(packed, np.uint32)
    sc = np.concatenate([b[..., 0:4] & 63, (b[..., 8:12] & 15) | ((b[..., 0:4] >> 6) << 4)], -1)
    mn = np.concatenate([b[..., 4:8] & 63, (b[..., 8:12] >> 4) | ((b[..., 4:8] >> 6) << 4)], -1)
    return sc.astype(np.uint8), mn.astype(np.uint8)


def _sub_planes(q, N, K):
    """q with its packed scales unpacked (test-side) into sc, mn [N][K/32]."""
    sc, mn = _unpack_k4(np.asarray(q["scales"]).reshape(N, K // 256, 12))
    return dict(q, sc=sc.reshape(N, K // 32), mn=mn.reshape(N, K // 32))


def test_q4_k_scale_packing():
    """The oracle's 12-byte packing of eight 6-bit scales and offsets against
    a worked example (bytes derived by hand from the layout) and against the
    test-side packer on random values; round trip; 4.5 bits per weight."""
    sc, mn = [1, 2, 3, 4, 48, 49, 50, 63], [5, 6, 7, 8, 33, 17, 62, 0]
    want = [193, 194, 195, 196, 133, 70, 199, 8, 16, 17, 226, 15]
    assert oracle.q4_k_pack_scales(sc, mn).tolist() == want
    assert _pack_k4(np.array(sc), np.array(mn)).tolist() == want
    got_sc, got_mn = oracle.q4_k_unpack_scales(np.array(want, np.uint8))
    assert got_sc.tolist() == sc and got_mn.tolist() == mn
    rng = np.random.default_rng(156)
    for _ in range(200):
        a, b = rng.integers(0, 64, 8), rng.integers(0, 64, 8)
        p = oracle.q4_k_pack_scales(a, b)
        assert np.array_equal(p, _pack_k4(a, b))
        ua, ub = _unpack_k4(p)
        assert np.array_equal(ua, a) and np.array_equal(ub, b)
    q = oracle.q4_k_quantize(synth.rand_bf16(157, (3, 512), 0.02), 3, 512)
    bits = 8 * sum(q[k].nbytes for k in ("qs", "scales", "d", "dmin"))
    assert bits == 4.5 * 3 * 512


def _q4_k_grid(q, N, K):
    """Per-weight step s = d*sc and offset o = dmin*mn, and the codes, as
    float64 arrays [N][K] (from the stored planes, not from the weights)."""
    q = _sub_planes(q, N, K)
    rep_sub = lambda a: np.repeat(a.astype(np.float64), 32, axis=1)
    rep_sup = lambda a: np.repeat(_f16(a).astype(np.float64), 256, axis=1)
    s = rep_sup(q["d"]) * rep_sub(q["sc"])
    o = rep_sup(q["dmin"]) * rep_sub(q["mn"])
    codes = np.empty((N, K), np.float64)
    codes[:, 0::2] = q["qs"] & 15
    codes[:, 1::2] = q["qs"] >> 4
    return s, o, codes


def _bf16_exact(v) -> bool:
    return float(bf16_to_f64(synth.to_bf16_bits(np.array([v], np.float32)))[0]) == v


def test_q4_k_exact_grid_round_trip():
    """Weights built as d*sc*q - dmin*m from chosen d = dmin = 2^-8, 6-bit
    sc and m (63 reached by both in every super-block) and 4-bit q (0 and
    15 reached in every sub-block), all exactly representable in bf16: the
    quantizer must give back exactly those planes and the decoder exactly
    those weights. Catches a wrong step (/15), a wrong super-scale (/63), a
    lost or sign-flipped offset, and swapped nibbles."""
    rng = np.random.default_rng(150)
    N, K = 6, 512
    h = 2.0 ** -8
    W = np.zeros((N, K), np.float32)
    want_sc = np.zeros((N, K // 32), np.uint8)
    want_mn = np.zeros((N, K // 32), np.uint8)
    want_q = np.zeros((N, K), np.uint8)
    for n in range(N):
        for sb in range(K // 256):
            j63, m63 = rng.choice(8, 2, replace=False)
            for j in range(8):
                while True:
                    sc = 63 if j == j63 else int(rng.integers(1, 64))
                    m = 63 if j == m63 else int(rng.integers(0, 64))
                    ok = [c for c in range(16) if _bf16_exact(h * (sc * c - m))]
                    if 0 in ok and 15 in ok and len(ok) >= 4:
                        break
                codes = rng.choice(ok, 32)
                codes[rng.choice(32, 2, replace=False)] = [0, 15]
                col = sb * 256 + j * 32
                W[n, col:col + 32] = h * (sc * codes - m)
                want_sc[n, col // 32], want_mn[n, col // 32] = sc, m
                want_q[n, col:col + 32] = codes
    B = synth.to_bf16_bits(W)
    assert np.array_equal(bf16_to_f64(B).reshape(N, K), W.astype(np.float64))
    q = _sub_planes(oracle.q4_k_quantize(B, N, K), N, K)
    assert np.all(_f16(q["d"]) == h) and np.all(_f16(q["dmin"]) == h)
    assert np.array_equal(q["sc"], want_sc) and np.array_equal(q["mn"], want_mn)
    assert np.array_equal(q["qs"], (want_q[:, 0::2] | (want_q[:, 1::2] << 4)).astype(np.uint8))
    assert np.array_equal(oracle.q4_k_dequantize(q, N, K), B)


def _q4_k_random_weights(seed, N, K):
    rng = np.random.default_rng(seed)
    W = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    W[:, rng.choice(K, K // 64, replace=False)] *= 12        # outlier channels
    W[: N // 4] += 0.01                                       # rows with a mean offset
    W[N // 4: N // 2] = np.abs(W[N // 4: N // 2])             # all-positive rows
    return synth.to_bf16_bits(W)


def test_q4_k_codes_are_nearest_on_the_stored_grid():
    """Brute force over the 16 codes: each stored code is a nearest grid point
    s*q - o of the stored grid (up to the binary32 rounding of (w + o)/s).
    Catches codes taken from the unrounded sub-block step, a wrong clamp
    range, and a flipped offset."""
    N, K = 64, 1024
    B = _q4_k_random_weights(151, N, K)
    q = oracle.q4_k_quantize(B, N, K)
    s, o, codes = _q4_k_grid(q, N, K)
    w = bf16_to_f64(B).reshape(N, K)
    err = np.abs(s * codes - o - w)
    best = np.min(np.abs(s[..., None] * np.arange(16.0) - o[..., None] - w[..., None]), axis=2)
    assert np.all(err <= best + s * 2.0 ** -20 + 1e-30)
    assert codes.max() == 15 and codes.min() == 0


def test_q4_k_error_bound_and_scale_ranges():
    """Every weight reads back within half a step plus what rounding the
    sub-block step to 6 bits of d can clip (15 * d/2) and what rounding the
    offset can shift (dmin/2), plus the bf16 rounding of the read-back
    value; 6-bit planes stay in [0, 63] and reach 62 or 63 in every
    super-block (d is max step / 63 up to binary16 rounding). Catches a
    floor in place of round-to-nearest for the 6-bit scales and offsets."""
    N, K = 64, 1024
    B = _q4_k_random_weights(152, N, K)
    q = _sub_planes(oracle.q4_k_quantize(B, N, K), N, K)
    s, o, _ = _q4_k_grid(q, N, K)
    w = bf16_to_f64(B).reshape(N, K)
    r = bf16_to_f64(oracle.q4_k_dequantize(q, N, K)).reshape(N, K)
    d = np.repeat(_f16(q["d"]).astype(np.float64), 256, axis=1)
    dm = np.repeat(_f16(q["dmin"]).astype(np.float64), 256, axis=1)
    bound = s / 2 + 7.5 * d + dm / 2 + np.abs(r) * 2.0 ** -8
    assert np.all(np.abs(r - w) <= bound * (1 + 2.0 ** -12))
    for plane in (q["sc"], q["mn"]):
        assert plane.max() <= 63
    tops = q["sc"].reshape(N, K // 256, 8).max(axis=2)
    assert np.all((tops == 63) | (tops == 62))
    # the all-positive rows need no offset: every sub-block minimum is >= 0
    assert not q["mn"][N // 4: N // 2].any() and not q["dmin"][N // 4: N // 2].any()


def test_q4_k_grid_spans_each_sub_block():
    """The stored grid reproduces each sub-block's span: its lowest point
    -dmin*m lies within dmin/2 of min(0, min w), its step d*sc within d/2 of
    (max w - min(0, min w)) / 15 (where the 6-bit values are below 63), and
    the largest step equals 63 d to binary16 precision. Catches rounding the
    6-bit offsets or scales down instead of to nearest."""
    N, K = 64, 1024
    B = _q4_k_random_weights(155, N, K)
    q = _sub_planes(oracle.q4_k_quantize(B, N, K), N, K)
    w = bf16_to_f64(B).reshape(N, K // 32, 32)
    lo = np.minimum(w.min(axis=2), 0.0)
    span = (w.max(axis=2) - lo) / 15
    d = np.repeat(_f16(q["d"]).astype(np.float64), 8, axis=1)
    dm = np.repeat(_f16(q["dmin"]).astype(np.float64), 8, axis=1)
    tol = 1 + 2.0 ** -10
    ok_m = q["mn"] < 63
    assert np.all(np.abs(-dm * q["mn"] - lo)[ok_m] <= (dm / 2 * tol)[ok_m])
    ok_s = q["sc"] < 63
    assert np.all(np.abs(d * q["sc"] - span)[ok_s] <= (d / 2 * tol)[ok_s])
    top = span.reshape(N, K // 256, 8).max(axis=2)
    assert np.allclose(63 * _f16(q["d"]).astype(np.float64), top, rtol=2.0 ** -10)


def test_q4_k_special_blocks():
    """A zero super-block (all planes 0, reads back 0); a constant negative
    sub-block (step 0, codes 0, read back as -dmin*m); a super-block whose
    step caps d at 65504 (codes clamp at 15 and 0)."""
    W = np.zeros((1, 768), np.float32)
    W[0, 256:288] = -0.75
    W[0, 288:512] = np.linspace(-0.5, 0.5, 224)
    W[0, 512] = 3.0e9
    W[0, 513] = -1.0e6
    B = synth.to_bf16_bits(W)
    q = _sub_planes(oracle.q4_k_quantize(B, 1, 768), 1, 768)
    r = bf16_to_f64(oracle.q4_k_dequantize(q, 1, 768))[0]
    assert q["d"][0, 0] == 0 and q["dmin"][0, 0] == 0
    assert not q["sc"][0, :8].any() and not q["mn"][0, :8].any() and not q["qs"][0, :128].any()
    assert not r[:256].any()
    assert q["sc"][0, 8] == 0 and not q["qs"][0, 128:144].any()
    assert abs(r[256] + 0.75) <= float(_f16(q["dmin"])[0, 1]) / 2
    assert _f16(q["d"])[0, 2] == 65504.0 and q["sc"][0, 16] == 63
    assert (q["qs"][0, 256] & 15) == 15 and (q["qs"][0, 256] >> 4) == 0


def test_q4_k_dequantize_is_binary32_then_bf16():
    """Read-back against torch's own conversions of the exact value
    d*sc*q - dmin*m (exact in binary64): binary64 -> binary32 -> bf16."""
    import torch
    rng = np.random.default_rng(153)
    N, K = 4, 512
    sc = rng.integers(0, 64, (N, K // 256, 8))
    mn = rng.integers(0, 64, (N, K // 256, 8))
    q = {"qs": rng.integers(0, 256, (N, K // 2)).astype(np.uint8),
         "scales": _pack_k4(sc, mn).reshape(N, K // 256 * 12),
         "d": np.array([[oracle.float_to_half(float(v)) for v in rng.lognormal(-7, 2, K // 256)]
                        for _ in range(N)], np.uint16),
         "dmin": np.array([[oracle.float_to_half(float(v)) for v in rng.lognormal(-7, 2, K // 256)]
                           for _ in range(N)], np.uint16)}
    s, o, codes = _q4_k_grid(q, N, K)
    exact = torch.from_numpy(s * codes - o)
    want = exact.to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.q4_k_dequantize(q, N, K), want)


def test_q4_k_linear_against_numpy_fp64():
    c = synth.linear_case([154], 33, 40, 512)
    q = oracle.q4_k_quantize(c["W"], 40, 512)
    Wd = oracle.q4_k_dequantize(q, 40, 512)
    Y = oracle.q4_k_linear(c["X"], q, c["bias"], 33, 40, 512)
    X = bf16_to_f64(c["X"]).reshape(33, 512)
    ref = X @ bf16_to_f64(Wd).reshape(40, 512).T + bf16_to_f64(c["bias"])[None, :]
    y = bf16_to_f64(Y).reshape(33, 40)
    assert np.all(np.abs(y - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-30)


# --------------------------------------------------------------------------
# adaLN modulation ahead of the activation quantization (Section 2: the
# modulation is generated at run time, so smoothing stays a runtime step)
# --------------------------------------------------------------------------

def _adaln_case(seed, M, K):
    rng = np.random.default_rng(seed)
    X = rng.normal(0, 1, (M, K)).astype(np.float32)
    X[:, rng.choice(K, max(1, K // 100), replace=False)] *= 20     # outlier channels
    X[M // 2:] += rng.normal(0, 3, (M - M // 2, 1)).astype(np.float32)   # row offsets
    shift = rng.normal(0, 0.05, K).astype(np.float32)
    scale = rng.normal(0, 0.1, K).astype(np.float32)
    return synth.to_bf16_bits(X), synth.to_bf16_bits(shift), synth.to_bf16_bits(scale)


def test_adaln_matches_torch_layer_norm_fp64():
    """Against torch's float64 layer_norm (its own mean, variance and eps
    handling), times (1 + scale) plus shift, rounded once to bf16 by exact
    rational rounding. Catches a sample variance, eps outside the root, a
    missing centering, '1 + scale' as 'scale', and shift/scale swapped."""
    import torch
    M, K = 12, 384
    X, shift, scale = _adaln_case(170, M, K)
    eps = 1e-6
    H = oracle.adaln_modulate(X, shift, scale, M, K, eps)
    x = torch.from_numpy(bf16_to_f64(X).reshape(M, K))
    ln = torch.nn.functional.layer_norm(x, (K,), eps=eps)
    ref = ln * (1 + torch.from_numpy(bf16_to_f64(scale))) + torch.from_numpy(bf16_to_f64(shift))
    want = np.array([[round_bf16_exact(float(v)) for v in row] for row in ref.numpy()], np.uint16)
    assert np.array_equal(H, want)


def test_adaln_special_rows_and_modulation():
    """A constant row normalizes to zero, so it reads back as bf16(shift)
    exactly; scale = -1 cancels the norm everywhere; with shift = scale = 0
    and eps = 0 every row has mean ~0 and population variance ~1."""
    M, K = 6, 256
    X, shift, scale = _adaln_case(171, M, K)
    Xc = X.copy()
    Xc[0] = Xc[0, 0]
    H = oracle.adaln_modulate(Xc, shift, scale, M, K, 1e-6)
    assert np.array_equal(H[0], shift)
    minus_one = np.full(K, 0xBF80, np.uint16)
    assert np.array_equal(oracle.adaln_modulate(X, shift, minus_one, M, K, 1e-6),
                          np.broadcast_to(shift, (M, K)))
    zero = np.zeros(K, np.uint16)
    h = bf16_to_f64(oracle.adaln_modulate(X, zero, zero, M, K, 0.0)).reshape(M, K)
    assert np.all(np.abs(h.mean(axis=1)) < 2e-3)
    assert np.allclose(h.var(axis=1), 1.0, atol=5e-3)


def test_adaln_eps_enters_under_the_root():
    """A row of +-a has variance a^2 exactly, so x - mean = +-a and the norm
    is a / sqrt(a^2 + eps): with a = 2^-10 and eps = 3 * 2^-20 it is exactly
    1/2 (no rounding anywhere)."""
    K = 64
    a = 2.0 ** -10
    X = synth.to_bf16_bits(np.tile(np.array([a, -a], np.float32), K // 2)[None, :])
    zero = np.zeros(K, np.uint16)
    h = bf16_to_f64(oracle.adaln_modulate(X, zero, zero, 1, K, 3 * 2.0 ** -20))
    assert np.array_equal(h.reshape(K), np.tile([0.5, -0.5], K // 2))


def test_adaln_quant_act_is_quant_act_of_the_modulated_row():
    M, K = 8, 256
    X, shift, scale = _adaln_case(172, M, K)
    il = np.random.default_rng(173).uniform(0.5, 2.0, K).astype(np.float32)
    Xq, xs = oracle.adaln_quant_act(X, shift, scale, il, M, K, 1e-6)
    H = bf16_to_f64(oracle.adaln_modulate(X, shift, scale, M, K, 1e-6)).reshape(M, K)
    v = (H.astype(np.float32) * il).astype(np.float64)
    amax = np.abs(v).max(axis=1)
    assert np.allclose(xs, amax / 127, rtol=2.0 ** -23)
    assert np.all(np.abs(Xq * xs[:, None].astype(np.float64) - v) <= xs[:, None] * QUANT_SLACK)
