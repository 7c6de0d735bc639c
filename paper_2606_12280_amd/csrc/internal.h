// Internal launchers of libw8a8 (not part of the ABI). Every launcher assumes
// its arguments were validated by the entry points in api.hip, enqueues on
// `stream` and returns the hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {

// Smoothing + per-row symmetric INT8 quantization of R rows of K bf16
// values: out[r][k] = clamp(rint((src[r][k] * mul[k]) * RN(127/absmax_r))),
// scale[r] = absmax_r / 127 (0 and all-zero codes below the tiny threshold).
hipError_t launch_smooth_quant_rows(const uint16_t *src, const float *mul,
                                    int64_t R, int64_t K, int8_t *out,
                                    float *scale, hipStream_t stream);

// inv[k] = RN(1 / lam[k]).
hipError_t launch_reciprocal(const float *lam, int64_t K, float *inv,
                             hipStream_t stream);

// colmax[k] = max(colmax[k], max_r |src[r][k]|) over R rows of bf16.
hipError_t launch_col_absmax(const uint16_t *src, int64_t R, int64_t K,
                             float *colmax, hipStream_t stream);

// Fragility statistics of the n bf16 entries of X (8 | n): stats[0..3] =
// max |x|, mean, population std, Pearson kurtosis (binary64). work holds
// 6 * kMomentBlocks doubles: each workgroup's count, mean, central sums of
// the second to fourth powers and max |x|.
constexpr int kMomentBlocks = 1024;
hipError_t launch_act_moments(const uint16_t *X, int64_t n, double *work, double *stats,
                              hipStream_t stream);
// The same with the workgroup states in the library's file-scope device
// array of the current device (no workspace, no allocation).
hipError_t launch_act_moments_noalloc(const uint16_t *X, int64_t n, double *stats,
                                      hipStream_t stream);

// GGUF Q8_0: codes qs [N][K] and binary16 scales d [N][K/32] of W [N][K]
// bf16 (32 | K), and back to bf16(d * q).
hipError_t launch_q8_0_quantize(const uint16_t *W, int64_t N, int64_t K, int8_t *qs,
                                uint16_t *d, hipStream_t stream);
hipError_t launch_q8_0_dequantize(const int8_t *qs, const uint16_t *d, int64_t N, int64_t K,
                                  uint16_t *W, hipStream_t stream);

// adaLN-modulated activation quantization: Xq, x_scale of
// quant_act(bf16(LayerNorm(X) * (1 + scale) + shift), inv_lambda), the norm
// in binary64 (64 | K, K <= 8192).
hipError_t launch_adaln_quant_act(const uint16_t *X, const uint16_t *shift,
                                  const uint16_t *scale, const float *inv_lambda, int64_t M,
                                  int64_t K, double eps, int8_t *Xq, float *x_scale,
                                  hipStream_t stream);

// GGUF Q4_K (256 | K): W [N][K] bf16 -> codes qs [N][K/2] (two per byte,
// even k low), the 6-bit sub-block scales and offsets packed 12 bytes per
// super-block in scales [N][K/256][12] (4-byte aligned), binary16
// super-block scales d and dmin [N][K/256]; and back to
// bf16(RN32(d * sc * q - dmin * mn)).
hipError_t launch_q4_k_quantize(const uint16_t *W, int64_t N, int64_t K, uint8_t *qs,
                                uint8_t *scales, uint16_t *d, uint16_t *dmin,
                                hipStream_t stream);
hipError_t launch_q4_k_dequantize(const uint8_t *qs, const uint8_t *scales, const uint16_t *d,
                                  const uint16_t *dmin, int64_t N, int64_t K, uint16_t *W,
                                  hipStream_t stream);

// dst[k] = 0 for k < K (a fill kernel, so that the call can be captured).
hipError_t launch_zero_f32(float *dst, int64_t K, hipStream_t stream);

// lam[k] = s[k]^alpha / lam[k]^(1-alpha) in binary64 (lam holds the weight
// column absmax on entry); 1 where either statistic is zero.
hipError_t launch_lambda_from_stats(const float *s, float *lam, int64_t K,
                                    double alpha, hipStream_t stream);

// C[m][n] = sum_k A[m][k] * B[n][k] with int8 operands; epilogue either
// stores the int32 sum (Y32 != nullptr) or bf16(acc * xs[m] * ws[n] + b[n]).
hipError_t launch_gemm_i8(const int8_t *A, const int8_t *B, const float *xs,
                          const float *ws, const uint16_t *bias, int64_t M,
                          int64_t N, int64_t K, uint16_t *Y, int32_t *Y32,
                          hipStream_t stream);

// Y[m][n] = bf16(sum_k A[m][k] * B[n][k] + b[n]) with bf16 operands and
// binary32 accumulation.
hipError_t launch_gemm_bf16(const uint16_t *A, const uint16_t *B,
                            const uint16_t *bias, int64_t M, int64_t N,
                            int64_t K, uint16_t *Y, hipStream_t stream);

// The tile (tokens x channels) and threads per workgroup of the GEMM the
// two launchers above run for M x N with K bytes per row (host only).
void gemm_config(int64_t M, int64_t N, int64_t Kb, int *tile_m, int *tile_n, int *threads);

}  // namespace w8a8
