/*
 * w8a8.h -- C ABI of the MI355X (gfx950) INT8 W8A8 quantized linear.
 *
 * The library implements the INT8 W8A8 recipe of "Quantizing a Dual-Branch
 * Flow-Matching Diffusion Transformer for Consumer GPUs" (arXiv 2606.12280),
 * Section 3, paragraphs "INT8 W8A8" and "Activation-fragility profiling and
 * protection":
 *   - weights: per-output-row (per-channel) symmetric INT8, round to nearest;
 *   - activations: per-token dynamic symmetric INT8;
 *   - SmoothQuant smoothing with lambda_j = s_j^alpha / max_i |W_ij|^(1-alpha)
 *     (weights scaled up by lambda, activations down);
 *   - the most fragile layers kept in bf16 with no activation quantization.
 *
 * Conventions shared by every entry point:
 *   - Matrices are row-major and packed: X [M][K] (M tokens, K input
 *     channels), W [N][K] (N output channels; the nn.Linear layout),
 *     Y [M][N]. bf16 values are passed as uint16_t bit patterns.
 *   - Every pointer is a DEVICE pointer owned by the caller. The library
 *     allocates nothing, keeps no state between calls and is re-entrant.
 *   - `stream` is a hipStream_t passed as an opaque pointer (NULL = the null
 *     stream). Every call only enqueues work on it and returns; inputs must
 *     stay alive and unmodified until the stream reaches the call.
 *   - Arguments are validated before any HIP call; on a validation error
 *     nothing is enqueued. A failed launch returns W8A8_ERR_HIP. Faults in
 *     the kernels surface at the caller's next synchronization.
 *   - Sizes: 1 <= M <= 2^22 rows (tokens; also N for the weight-side row
 *     kernels; fewer than 2^22 when K > 32768, W8A8_ERR_SHAPE otherwise);
 *     an empty token batch, M = 0, is accepted by every entry point that
 *     takes tokens except w8a8_act_moments (no statistics of no entries):
 *     the other arguments are validated as usual, buffers sized by M may
 *     then be NULL, W8A8_OK is returned and nothing is enqueued (q8_0_linear
 *     and q4_k_linear then leave `work` untouched);
 *     GEMM outputs 1 <= N <= 2^20 and M * N <= 2^38;
 *     64 <= K <= 65536 with K % 64 == 0 (the int32 sum is then exact:
 *     127^2 * K < 2^31). Ragged M and N need no padding. Matrix pointers
 *     and lambda / inv_lambda must be 16-byte aligned; scales 4-byte and
 *     bias 2-byte aligned. Outputs may not overlap inputs.
 *   - Inputs must be finite. Results are deterministic: the same inputs give
 *     the same bits on every call.
 *   - Codes and scales use binary32 arithmetic with one IEEE rounding per
 *     operation: x' = x * inv_lambda, absmax, scale = absmax / 127,
 *     code = clamp(rint(x' * RN(127 / absmax)), -127, 127) with rint = round
 *     half to even. A row whose absmax is below 2^-96 (including an all-zero
 *     row) gets scale 0 and all-zero codes.
 */
#ifndef W8A8_H
#define W8A8_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum w8a8_status {
    W8A8_OK = 0,
    W8A8_ERR_NULL = 1,        /* a required pointer is NULL */
    W8A8_ERR_SHAPE = 2,       /* a size is out of range */
    W8A8_ERR_ALIGN = 3,       /* a pointer is not aligned as required */
    W8A8_ERR_ALIAS = 4,       /* an output overlaps an input or another output */
    W8A8_ERR_UNSUPPORTED = 5, /* a valid request this library does not handle
                                 (K not a multiple of 64, K > 65536, alpha
                                 outside (0, 1)) */
    W8A8_ERR_HIP = 6          /* the HIP runtime reported an error */
} w8a8_status;

/* Opaque hipStream_t. */
typedef void *w8a8_stream;

/* Version of this ABI (increases on any incompatible change). */
int w8a8_abi_version(void);

/* Static description of a status code; never NULL. */
const char *w8a8_status_string(int status);

/* Name of the last HIP error seen by a call that returned W8A8_ERR_HIP on the
 * calling thread ("" if none). */
const char *w8a8_last_hip_error(void);

/* ---------------------------------------------------------------------- */
/* Calibration (Section 3, "INT8 W8A8": the per-channel activation scales */
/* are measured beforehand on calibration inputs; the smoothing equation).*/
/* ---------------------------------------------------------------------- */

/* Per-input-channel activation absmax, accumulated:
 *   absmax[k] = max(absmax[k], max_t |X[t][k]|)        for k < K.
 * X [M][K] bf16; absmax [K] fp32, read and written (seed it with zeros for a
 * fresh pass; call again per calibration batch). */
w8a8_status w8a8_act_absmax(const uint16_t *X, int64_t M, int64_t K,
                            float *absmax, w8a8_stream stream);

/* Fragility profile of one linear's input for one denoising step
 * (Section 3, "Activation-fragility profiling and protection": max-abs,
 * standard deviation and kurtosis per layer and step). Over the n = M*K
 * entries of X [M][K] bf16, with mean = (1/n) sum x and
 * m_j = (1/n) sum (x - mean)^j, writes four binary64 values:
 *   stats[0] = max |x|, stats[1] = mean, stats[2] = sqrt(m2) (population
 *   standard deviation), stats[3] = m4 / m2^2 (Pearson kurtosis, 3 for a
 *   Gaussian; 0 when m2 == 0).
 * One pass over X: central moments of groups of entries, merged pairwise in
 * a fixed grid and a fixed order, so equal inputs give equal bits. work: device
 * scratch of W8A8_MOMENTS_WORK_BYTES bytes owned by the caller, 8-byte
 * aligned, overwritten; calls that share it must be ordered on one stream.
 * stats: device, 4 doubles, 8-byte aligned. Same M and K limits as the other
 * calls (K % 64 == 0). */
#define W8A8_MOMENTS_WORK_BYTES (6 * 1024 * 8)
w8a8_status w8a8_act_moments(const uint16_t *X, int64_t M, int64_t K, void *work,
                             double *stats, w8a8_stream stream);

/* w8a8_act_moments for callers that cannot allocate device memory or pass
 * a workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels, results bit-identical to
 * w8a8_act_moments on the same X, with the workgroup states in a
 * W8A8_MOMENTS_WORK_BYTES device array that the library itself holds, one
 * per GPU, from that GPU's first call until the process ends. That array is
 * a fixed size for every input, so the limits are those of
 * w8a8_act_moments (M and K out of range: W8A8_ERR_SHAPE or
 * W8A8_ERR_UNSUPPORTED). The call allocates nothing; its first call on a
 * device looks the array's address up (hipGetSymbolAddress), so the device
 * of X, stats and stream must be the current device. Nothing in the array
 * needs to start at zero. Calls on one GPU share the array: calls that can
 * overlap there (different streams without ordering) race and give wrong
 * statistics; order them on one stream. */
w8a8_status w8a8_act_moments_noalloc(const uint16_t *X, int64_t M, int64_t K,
                                     double *stats, w8a8_stream stream);

/* Protection choice (Section 3, "Activation-fragility profiling and
 * protection": the layers whose inputs are most fragile stay in bf16, N = 17
 * of 211 per branch, and the ranking is checked for stability between the
 * early and late halves of the trajectory). The paper gives no formula for
 * the score; a layer's score here is its input kurtosis averaged over the
 * profiled steps. These three are HOST functions: every pointer is host
 * memory, nothing is launched and no GPU is needed. Inputs must be finite,
 * else W8A8_ERR_UNSUPPORTED; at most 2^20 layers and 2^20 steps.
 *
 * Scores: kurtosis [layers][steps] binary64 (row-major, e.g. stats[3] of
 * w8a8_act_moments per layer and step) -> scores [layers], the sum over
 * steps step_begin <= s < step_end in step order divided by the number of
 * those steps (0 <= step_begin < step_end <= steps). */
w8a8_status w8a8_fragility_scores(const double *kurtosis, int64_t layers,
                                  int64_t steps, int64_t step_begin,
                                  int64_t step_end, double *scores);

/* The n most fragile layers: indices [n] of the n highest of scores
 * [layers], highest first, equal scores in increasing layer index
 * (0 <= n <= layers; indices may be NULL when n == 0). */
w8a8_status w8a8_select_protected(const double *scores, int64_t layers,
                                  int64_t n, int32_t *indices);

/* Spearman rank correlation of a [n] and b [n] (n >= 2): the Pearson
 * correlation of their 1-based ranks, equal values sharing the mean of their
 * positions. A constant vector has no ranking: W8A8_ERR_UNSUPPORTED. */
w8a8_status w8a8_rank_correlation(const double *a, const double *b, int64_t n,
                                  double *rho);

/* SmoothQuant factors (Section 3, the smoothing equation):
 *   lambda[j] = act_absmax[j]^alpha / (max_i |W[i][j]|)^(1 - alpha),
 * computed in binary64 (sqrt(s)/sqrt(m) when alpha == 0.5, else
 * pow(s, alpha) / pow(m, 1 - alpha)) and rounded once to binary32. A channel
 * whose activation absmax or weight-column absmax is 0 gets lambda = 1.
 * act_absmax [K] fp32, W [N][K] bf16 -> lambda [K] fp32 (also used as the
 * kernel's scratch for the column absmax). 0 < alpha < 1. */
w8a8_status w8a8_smooth_factors(const float *act_absmax, const uint16_t *W,
                                int64_t N, int64_t K, double alpha,
                                float *lambda, w8a8_stream stream);

/* ---------------------------------------------------------------------- */
/* The quantized linear (Section 3, "INT8 W8A8").                          */
/* ---------------------------------------------------------------------- */

/* Offline weight preparation, once per layer:
 *   inv_lambda[k] = RN(1 / lambda[k]);
 *   W'[n][k] = W[n][k] * lambda[k];  per output row n: s = absmax/127 and
 *   Wq[n][k] = clamp(rint(W'[n][k] * RN(127/absmax)), -127, 127).
 * W [N][K] bf16, lambda [K] fp32 (finite, > 0) -> Wq [N][K] int8,
 * w_scale [N] fp32, inv_lambda [K] fp32 (consumed by w8a8_quant_act).
 * Pass lambda = all ones for a layer without smoothing. */
w8a8_status w8a8_prepare_weight(const uint16_t *W, const float *lambda,
                                int64_t N, int64_t K, int8_t *Wq,
                                float *w_scale, float *inv_lambda,
                                w8a8_stream stream);

/* Runtime activation path, steps (1) smooth and (2) quantize per token:
 *   X'[t][k] = X[t][k] * inv_lambda[k];  per token t: s = absmax/127 and
 *   Xq[t][k] = clamp(rint(X'[t][k] * RN(127/absmax)), -127, 127).
 * X [M][K] bf16, inv_lambda [K] fp32 -> Xq [M][K] int8, x_scale [M] fp32.
 * One pass over X; the smoothed values never leave registers. */
w8a8_status w8a8_quant_act(const uint16_t *X, const float *inv_lambda,
                           int64_t M, int64_t K, int8_t *Xq, float *x_scale,
                           w8a8_stream stream);

/* The same activation step on the adaLN-modulated input of a DiT block's QKV
 * or FFN-up projection (Section 2: the modulation is generated at run time,
 * which is why smoothing is applied at run time), fused so that the
 * modulated tensor never goes to memory. Per token row t, in binary64:
 *   mean = sum_k X[t][k] / K,  var = sum_k (X[t][k] - mean)^2 / K,
 *   rstd = 1 / sqrt(var + eps),
 *   H[t][k] = bf16(((X[t][k] - mean) * rstd) * (1 + scale[k]) + shift[k])
 * (LayerNorm without affine terms, one rounding to bf16); then
 * exactly w8a8_quant_act(H, inv_lambda). X [M][K], shift [K], scale [K]
 * bf16, inv_lambda [K] fp32 -> Xq [M][K] int8, x_scale [M] fp32. K must be
 * a multiple of 64 and at most 8192 (the DiT's modulated inputs have
 * K = 4096), eps finite and >= 0, else
 * W8A8_ERR_UNSUPPORTED. Alignment as w8a8_quant_act, shift and scale
 * 16-byte aligned. */
w8a8_status w8a8_adaln_quant_act(const uint16_t *X, const uint16_t *shift,
                                 const uint16_t *scale, const float *inv_lambda,
                                 int64_t M, int64_t K, double eps, int8_t *Xq,
                                 float *x_scale, w8a8_stream stream);

/* Steps (3) INT8 GEMM and (4) fused epilogue:
 *   acc[t][n] = sum_k Xq[t][k] * Wq[n][k]   (exact int32),
 *   Y[t][n]   = bf16_rne(float(acc) * (x_scale[t] * w_scale[n]) + bias[n])
 * with the product and the bias add in binary32 (one fused multiply-add).
 * Xq [M][K] int8, x_scale [M], Wq [N][K] int8, w_scale [N], bias [N] bf16 or
 * NULL (no bias) -> Y [M][N] bf16. The int32 accumulators stay in registers. */
w8a8_status w8a8_linear(const int8_t *Xq, const float *x_scale,
                        const int8_t *Wq, const float *w_scale,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y, w8a8_stream stream);

/* The same GEMM main loop with the int32 accumulators stored instead of the
 * epilogue (for verification): C[t][n] = sum_k Xq[t][k] * Wq[n][k].
 * Xq [M][K] int8, Wq [N][K] int8 -> C [M][N] int32. */
w8a8_status w8a8_gemm_i32(const int8_t *Xq, const int8_t *Wq, int64_t M,
                          int64_t N, int64_t K, int32_t *C,
                          w8a8_stream stream);

/* Protected layer (Section 3: the top-N fragile layers stay in bf16 with no
 * activation quantization):
 *   Y[t][n] = bf16_rne(sum_k X[t][k] * W[n][k] + bias[n])
 * with bf16 products accumulated in binary32 (MFMA). X [M][K] bf16,
 * W [N][K] bf16 (the original, unsmoothed weights), bias [N] bf16 or NULL
 * -> Y [M][N] bf16. */
w8a8_status bf16_linear(const uint16_t *X, const uint16_t *W,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y, w8a8_stream stream);

/* Diagnostic, host only (launches nothing, needs no GPU): the GEMM
 * configuration that w8a8_linear and w8a8_gemm_i32 (bf16 == 0) or
 * bf16_linear (bf16 != 0) launch for an M x N x K problem: the output tile
 * of one workgroup, tile_m tokens x tile_n channels, and its threads.
 * The same shape checks as those entry points (W8A8_ERR_SHAPE,
 * W8A8_ERR_UNSUPPORTED); NULL outputs give W8A8_ERR_NULL. */
w8a8_status w8a8_gemm_config(int64_t M, int64_t N, int64_t K, int bf16,
                             int32_t *tile_m, int32_t *tile_n, int32_t *threads);

/* ---------------------------------------------------------------------- */
/* GGUF Q8_0 weight-only (Section 3, "GGUF k-quants": 8.5 bits per weight, */
/* round to nearest). A row of W [N][K] is cut into blocks of 32           */
/* consecutive weights; a block keeps 32 int8 codes and a binary16 scale.  */
/* Stored planar: qs [N][K] int8 and d [N][K/32] binary16 bits.            */
/* ---------------------------------------------------------------------- */

/* Encode, per block: amax = max |w|, d = RN16(min(RN32(amax / 127), 65504)),
 * q = clamp(rint(w * RN32(1 / float(d))), -127, 127) (all 0 if d == 0), in
 * binary32 with one rounding per operation. W [N][K] bf16 (16-byte aligned)
 * -> qs [N][K] int8 (16-byte aligned), d [N][K/32] (2-byte aligned). Same N
 * and K limits as w8a8_prepare_weight (K % 64 == 0). */
w8a8_status q8_0_quantize(const uint16_t *W, int64_t N, int64_t K, int8_t *qs,
                          uint16_t *d, w8a8_stream stream);

/* Decode: W[n][k] = bf16_rne(float(d[n][k/32]) * qs[n][k]) (the product is
 * exact in binary32). qs, d as above -> W [N][K] bf16 (16-byte aligned). */
w8a8_status q8_0_dequantize(const int8_t *qs, const uint16_t *d, int64_t N,
                            int64_t K, uint16_t *W, w8a8_stream stream);

/* The weight-only linear: Y = bf16_linear(X, decode(qs, d), bias), i.e.
 *   Y[t][n] = bf16_rne(sum_k X[t][k] * W'[n][k] + bias[n]), W' = decode(qs, d),
 * bf16 products accumulated in binary32. The decoded weights go to `work`
 * (caller-owned, 2 N K bytes, 16-byte aligned, overwritten): weights stay
 * resident at 8.5 bits per weight and only the layer being run is decoded.
 * X [M][K] bf16, bias [N] bf16 or NULL -> Y [M][N] bf16. Same limits as
 * bf16_linear. */
w8a8_status q8_0_linear(const uint16_t *X, const int8_t *qs, const uint16_t *d,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K,
                        uint16_t *work, uint16_t *Y, w8a8_stream stream);

/* ---------------------------------------------------------------------- */
/* GGUF Q4_K weight-only (Section 3, "GGUF k-quants": 4-bit codes in       */
/* super-blocks, 4.5 bits per weight; the encoder is the paper's own). A   */
/* super-block is 256 consecutive weights of a row, cut into 8 sub-blocks  */
/* of 32; sub-block j reads back as d*sc_j*q - dmin*m_j with q in [0,15],  */
/* sc_j, m_j in [0,63] and binary16 d, dmin per super-block. Stored planar: */
/*   qs [N][K/2]  two 4-bit codes per byte, even k in the low nibble       */
/*   scales [N][K/256][12]  the super-block's sc_j and m_j in the GGUF     */
/*     k-quant scale layout: for j < 4, bytes j and j+4 hold sc_j and m_j  */
/*     in their low 6 bits; for j >= 4, byte j+4 holds the low 4 bits of   */
/*     sc_j (low nibble) and m_j (high nibble), and their top 2 bits are   */
/*     the top 2 bits of bytes j-4 (sc_j) and j (m_j)                      */
/*   d, dmin [N][K/256]  binary16 bits                                     */
/* (4 + (96 + 32)/256 = 4.5 bits per weight). K must be a multiple of 256, */
/* else W8A8_ERR_UNSUPPORTED; qs 16-byte aligned, scales 4-byte, d and     */
/* dmin 2-byte aligned.                                                    */
/* ---------------------------------------------------------------------- */

/* Encode, round to nearest on a min-max grid (binary32, one rounding per
 * operation): per sub-block lo = min(0, min w), hi = max w,
 * a_j = (hi - lo)/15, b_j = -lo; d = RN16(min(max_j a_j/63, 65504)) and
 * dmin likewise from the b_j; sc_j = min(rint(a_j*RN32(1/d)), 63),
 * m_j = min(rint(b_j*RN32(1/dmin)), 63) (0 where d or dmin is 0); codes
 * q = clamp(rint((w + dmin*m_j)*RN32(1/(d*sc_j))), 0, 15) (0 where d*sc_j
 * is 0). W [N][K] bf16, 16-byte aligned. Outputs must not overlap W or
 * each other. */
w8a8_status q4_k_quantize(const uint16_t *W, int64_t N, int64_t K, uint8_t *qs,
                          uint8_t *scales, uint16_t *d, uint16_t *dmin,
                          w8a8_stream stream);

/* Decode: W[n][k] = bf16(RN32(d*sc_j*q - dmin*m_j)) (d*sc_j*q is exact in
 * binary32). W [N][K] bf16, 16-byte aligned, must not overlap the planes. */
w8a8_status q4_k_dequantize(const uint8_t *qs, const uint8_t *scales,
                            const uint16_t *d, const uint16_t *dmin, int64_t N,
                            int64_t K, uint16_t *W, w8a8_stream stream);

/* The weight-only linear on the decoded weights: Y = bf16_linear(X,
 * decode(planes), bias). The decoded weights go to `work` (caller-owned,
 * 2 N K bytes, 16-byte aligned, overwritten). X [M][K] bf16, bias [N] bf16
 * or NULL -> Y [M][N] bf16; limits as bf16_linear. */
w8a8_status q4_k_linear(const uint16_t *X, const uint8_t *qs, const uint8_t *scales,
                        const uint16_t *d, const uint16_t *dmin, const uint16_t *bias,
                        int64_t M, int64_t N, int64_t K, uint16_t *work, uint16_t *Y,
                        w8a8_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* W8A8_H */
