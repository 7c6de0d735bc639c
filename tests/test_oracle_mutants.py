"""Plants one mistake at a time in a copy of the CPU oracle and checks that the
pins in test_oracle_pins.py catch it (CPU only; nothing runs on a GPU).

Each mutant is a plausible slip in following the paper's Section 3 recipe: the
smoothing direction, the rounding rule, the scale, the SmoothQuant exponent, a
dropped bias, a wrong index. Clamping at -128 instead of -127 is not listed:
with scale = absmax/127 and code = rint(x * RN(127/absmax)) the clamp never
fires (|x * RN(127/absmax)| <= 127 + 2^-17 rounds to 127), so that mutant
computes the same codes."""
from __future__ import annotations

import os
import subprocess
import tempfile

import pytest

import oracle
import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "smoothing_direction": ("inv_lambda[k] = 1.0f / lambda[k];", "inv_lambda[k] = lambda[k];"),
    "weights_divided": ("smooth_quantize_row(W + n * K, lambda, K,",
                        "smooth_quantize_row(W + n * K, inv_lambda, K,"),
    "round_half_away": ("float c = rintf(v * r);", "float c = roundf(v * r);"),
    "scale_over_128": ("*scale = amax / 127.0f;", "*scale = amax / 128.0f;"),
    "reciprocal_128": ("r = 127.0f / amax;", "r = 128.0f / amax;"),
    "absmax_signed": ("float a = fabsf(bf16_to_float(src[k]) * mul[k]);",
                      "float a = bf16_to_float(src[k]) * mul[k];"),
    "tiny_row_rule": ("#define ORACLE_TINY_ABSMAX 0x1p-96f", "#define ORACLE_TINY_ABSMAX 0x1p-140f"),
    "alpha_swapped": ("pow(s, alpha) / pow(wmax, 1.0 - alpha)", "pow(s, 1.0 - alpha) / pow(wmax, alpha)"),
    "sqrt_inverted": ("(float)(sqrt(s) / sqrt(wmax))", "(float)(sqrt(wmax) / sqrt(s))"),
    "calib_signed": ("float a = fabsf(bf16_to_float(X[t * K + k]));", "float a = bf16_to_float(X[t * K + k]);"),
    "gemm_unsigned_x": ("acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            C[t * N + n]",
                        "acc += (int32_t)(uint8_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            C[t * N + n]"),
    "gemm_drops_last_k": ("for (k = 0; k < K; ++k)\n                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            C[t * N + n]",
                          "for (k = 0; k < K - 1; ++k)\n                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            C[t * N + n]"),
    "epilogue_drops_bias": ("double b = bias ? (double)bf16_to_float(bias[n]) : 0.0;\n            double y = (double)C",
                            "double b = 0.0;\n            double y = (double)C"),
    "epilogue_scale_index": ("((double)x_scale[t] * (double)w_scale[n]) + b;\n            Y[t * N + n] = double_to_bf16(y);\n        }\n}\n\n/* The W8A8",
                             "((double)x_scale[t] * (double)w_scale[t % N]) + b;\n            Y[t * N + n] = double_to_bf16(y);\n        }\n}\n\n/* The W8A8"),
    "bf16_double_rounding": ("q = nearbyint(ldexp(d, -ulp_exp));", "q = nearbyint(ldexp((double)(float)d, -ulp_exp));"),
    "bf16_subnormal_spacing": ("ulp_exp = -133;", "ulp_exp = -126;"),
    "protected_drops_bias": ("            if (bias)\n                acc += (double)bf16_to_float(bias[n]);\n", ""),
    "moments_sample_std": ("out[2] = sqrt(m2);", "out[2] = sqrt(s2 / (n - 1.0));"),
    "moments_excess_kurtosis": ("out[3] = m2 > 0.0 ? m4 / (m2 * m2) : 0.0;",
                                "out[3] = m2 > 0.0 ? m4 / (m2 * m2) - 3.0 : 0.0;"),
    "moments_not_centered": ("double d = (double)bf16_to_float(X[t * K + k]) - mean;",
                             "double d = (double)bf16_to_float(X[t * K + k]);"),
    "moments_signed_max": ("if (fabsf(x) > m)\n                m = fabsf(x);", "if (x > m)\n                m = x;"),
    "half_truncates": ("q = nearbyint(ldexp(fabs(d), -ulp_exp));", "q = floor(ldexp(fabs(d), -ulp_exp));"),
    "half_no_subnormals": ("    if (ulp_exp < -24)\n        ulp_exp = -24;\n    q = nearbyint(ldexp(fabs(d), -ulp_exp));",
                           "    if (ulp_exp < -14)\n        ulp_exp = -14;\n    q = nearbyint(ldexp(fabs(d), -ulp_exp));"),
    # coding against the unrounded scale is what the common GGUF encoder
    # does; under this repository's reading (codes on the stored grid) it is
    # a deviation the pins must notice, not a claim that the encoder is wrong
    "q8_0_codes_from_unrounded_scale": ("inv = ds != 0.0f ? 1.0f / ds : 0.0f;", "inv = s != 0.0f ? 1.0f / s : 0.0f;"),
    "q8_0_no_clamp": ("                if (c > 127.0f)\n                    c = 127.0f;\n", ""),
    "q8_0_no_scale_cap": ("            if (s > ORACLE_HALF_MAX)\n                s = ORACLE_HALF_MAX;\n", ""),
    "q8_0_dequant_drops_scale": ("float v = half_to_float(d[n * (K / ORACLE_Q8_0_BLOCK) + k / ORACLE_Q8_0_BLOCK]) *\n                      (float)qs[n * K + k];",
                                 "float v = (float)qs[n * K + k];"),
    "q4_k_nibbles_swapped": ("(uint8_t)(codes[k] | (codes[k + 1] << 4));", "(uint8_t)(codes[k + 1] | (codes[k] << 4));"),
    "q4_k_offset_sign": ("float c = rintf((bf16_to_float(w[j * ORACLE_Q4_K_SUB + i]) + o) * inv);",
                         "float c = rintf((bf16_to_float(w[j * ORACLE_Q4_K_SUB + i]) - o) * inv);"),
    "q4_k_codes_from_unrounded_step": ("inv = s != 0.0f ? 1.0f / s : 0.0f;\n        for (i = 0;",
                                       "inv = a[j] != 0.0f ? 1.0f / a[j] : 0.0f;\n        for (i = 0;"),
    "q4_k_scale_floor": ("float cs = rintf(a[j] * inv_d)", "float cs = floorf(a[j] * inv_d)"),
    "q4_k_offset_floor": ("cm = rintf(b[j] * inv_dm)", "cm = floorf(b[j] * inv_dm)"),
    "q4_k_super_scale_over_64": ("*d = float_to_half(cap_half(amax / 63.0f));", "*d = float_to_half(cap_half(amax / 64.0f));"),
    "q4_k_step_over_16": ("a[j] = (hi - lo) / 15.0f;", "a[j] = (hi - lo) / 16.0f;"),
    "q4_k_min_not_clamped_to_zero": ("float lo = 0.0f, hi = -INFINITY;", "float lo = INFINITY, hi = -INFINITY;"),
    "q4_k_pack_high_bits_shift": ("out[j - 4] |= (uint8_t)((sc[j] >> 4) << 6);",
                                  "out[j - 4] |= (uint8_t)((sc[j] >> 2) << 6);"),
    "q4_k_unpack_offset_nibble": ("mn[j] = (uint8_t)((in[j + 4] >> 4) | ((in[j] >> 6) << 4));",
                                  "mn[j] = (uint8_t)((in[j + 4] & 15) | ((in[j] >> 6) << 4));"),
    "q4_k_decode_drops_offset": ("v = s * q - o;", "v = s * q;"),
    "q4_k_no_code_clamp": ("            if (c > 15.0f)\n                c = 15.0f;\n", ""),
    "adaln_sample_variance": ("rstd = 1.0 / sqrt(ss / (double)K + eps);", "rstd = 1.0 / sqrt(ss / (double)(K - 1) + eps);"),
    "adaln_eps_outside_root": ("rstd = 1.0 / sqrt(ss / (double)K + eps);", "rstd = 1.0 / (sqrt(ss / (double)K) + eps);"),
    "adaln_scale_without_one": ("const double m = n * (1.0 + (double)bf16_to_float(scale[k]));",
                                "const double m = n * (double)bf16_to_float(scale[k]);"),
    "adaln_shift_scale_swapped": ("const double m = n * (1.0 + (double)bf16_to_float(scale[k]));\n            H[t * K + k] = double_to_bf16(m + (double)bf16_to_float(shift[k]));",
                                  "const double m = n * (1.0 + (double)bf16_to_float(shift[k]));\n            H[t * K + k] = double_to_bf16(m + (double)bf16_to_float(scale[k]));"),
    "adaln_uncentered_variance": ("const double c = (double)bf16_to_float(x[k]) - mean;", "const double c = (double)bf16_to_float(x[k]);"),
    "adaln_not_centered": ("const double n = ((double)bf16_to_float(x[k]) - mean) * rstd;", "const double n = (double)bf16_to_float(x[k]) * rstd;"),
    "linear_drops_last_k": ("for (k = 0; k < K; ++k)\n                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            y = (double)acc",
                            "for (k = 0; k + 1 < K; ++k)\n                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            y = (double)acc"),
    "linear_drops_bias": ("double b = bias ? (double)bf16_to_float(bias[n]) : 0.0;\n            double y;",
                          "double b = 0.0;\n            double y;"),
    "linear_scale_index": ("y = (double)acc * ((double)x_scale[t] * (double)w_scale[n]) + b;",
                           "y = (double)acc * ((double)x_scale[t] * (double)w_scale[t]) + b;"),
    "linear_transposed_weight": ("acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];\n            y = (double)acc",
                                 "acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[k * N + n];\n            y = (double)acc"),
    "moments_drops_last_row": ("    for (t = 0; t < M; ++t) {\n        s2 += r2[t];",
                               "    for (t = 0; t + 1 < M; ++t) {\n        s2 += r2[t];"),
}

# every pin, with fixed arguments for the parametrized ones
PINS = [
    pins.test_bf16_widening_matches_bit_layout,
    pins.test_double_to_bf16_matches_exact_rounding,
    lambda: pins.test_gemm_i32_matches_numpy_int64(17, 9, 128, 2),
    pins.test_gemm_i32_extreme_magnitudes,
    pins.test_act_absmax_matches_numpy_and_accumulates,
    pins.test_smooth_factors_closed_forms,
    lambda: pins.test_smoothing_balances_channel_ranges(0.25),
    pins.test_inv_lambda_is_correctly_rounded_reciprocal,
    pins.test_round_half_even_ties,
    pins.test_activation_quant_invariants_tiny,
    pins.test_weight_quant_invariants_tiny,
    pins.test_quant_special_rows,
    pins.test_lossless_grid_reduces_to_plain_product,
    lambda: pins.test_w8a8_error_bound_vs_fp64("tiny"),
    pins.test_epilogue_against_exact_rationals,
    pins.test_w8a8_linear_against_int64_and_exact_rationals,
    pins.test_bf16_linear_small_integers_exact,
    pins.test_bf16_linear_random_vs_numpy_fp64,
    pins.test_act_moments_against_exact_rationals,
    pins.test_act_moments_two_point_and_constant,
    pins.test_act_moments_shift_and_scale,
    pins.test_act_moments_matches_scipy,
    pins.test_half_conversion_matches_numpy,
    pins.test_q8_0_invariants,
    pins.test_q8_0_exact_grid_and_ties,
    pins.test_q8_0_special_blocks,
    pins.test_q8_0_dequantize_is_one_rounding,
    pins.test_adaln_matches_torch_layer_norm_fp64,
    pins.test_adaln_special_rows_and_modulation,
    pins.test_adaln_eps_enters_under_the_root,
    pins.test_q4_k_scale_packing,
    pins.test_q4_k_exact_grid_round_trip,
    pins.test_q4_k_codes_are_nearest_on_the_stored_grid,
    pins.test_q4_k_error_bound_and_scale_ranges,
    pins.test_q4_k_grid_spans_each_sub_block,
    pins.test_q4_k_special_blocks,
    pins.test_q4_k_dequantize_is_binary32_then_bf16,
]


def _caught() -> int:
    n = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            n += 1
    return n


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    before, after = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(before) == 1, "mutation site moved"
    c_path = tmp_path / "oracle_mut.c"
    c_path.write_text(src.replace(before, after))
    so_path = str(tmp_path / "liboracle_mut.so")
    subprocess.run(["gcc", *oracle.CFLAGS, "-w", "-o", so_path, str(c_path), "-lm"], check=True)
    oracle.use_library(so_path)
    try:
        caught = _caught()
    finally:
        oracle.use_library(None)
    assert caught >= 1, f"no pin catches the '{name}' mutant"


def test_unmutated_oracle_passes_every_pin():
    oracle.use_library(None)
    assert _caught() == 0
