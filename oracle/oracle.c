/*
 * oracle.c -- plain, slow CPU reference of the INT8 W8A8 quantized linear.
 *
 * TEST INFRASTRUCTURE. Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py load this library. The product library
 * (paper_2606_12280_amd/) never calls it, and the two share no source,
 * header, helper or table.
 *
 * It follows the recipe of Section 3 ("INT8 W8A8" and "Activation-fragility
 * profiling and protection") step by step, in the paper's order:
 *
 *   lambda_j = s_j^alpha / max_i |W_ij|^(1-alpha)      (the smoothing equation)
 *   weights multiplied by lambda, activations divided by lambda (SmoothQuant)
 *   weights: symmetric INT8 per output row, round to nearest (Section 2 notes
 *            that plain round-to-nearest suffices at 8 bits)
 *   activations: symmetric INT8 per token, scale computed on the fly
 *   int8 x int8 products summed exactly in int32
 *   rescale by s_tok * s_ch, add the bias, round once to bf16
 *   protected layers: bf16 X times bf16 W^T plus bias, no smoothing and no
 *            activation quantization
 *
 * Readings of points the paper leaves open (each one is listed, with its
 * reason, in the design notes of the repository):
 *   - every scalar of the quantization is binary32, one IEEE rounding per
 *     operation, no fused multiply-add; the quantized codes depend on it, so
 *     the GPU takes the same decisions in the same precision;
 *   - "divide by lambda" is a multiply by inv_lambda = RN(1/lambda), computed
 *     once per input channel;
 *   - scale = absmax/127 and code = clamp(rint(x * RN(127/absmax)), -127, 127)
 *     with rint = round half to even; -128 is never produced;
 *   - a row (token or output channel) whose absmax is below 2^-96, including
 *     an all-zero row, gets scale 0 and all-zero codes, so that 127/absmax
 *     never overflows;
 *   - the epilogue and the protected linear are computed in binary64 and
 *     rounded once to bf16 (round to nearest even);
 *   - lambda itself is computed in binary64 and rounded once to binary32; a
 *     channel whose activation or weight statistic is zero keeps lambda = 1;
 *   - the fragility profile of a layer's input is max |x|, the population
 *     standard deviation and the Pearson kurtosis m4 / m2^2 over all its
 *     entries, in binary64; a constant input has kurtosis 0;
 *   - GGUF Q8_0 (Section 3, "GGUF k-quants"): blocks of 32 consecutive
 *     weights of a row; d = RN16(min(RN32(amax / 127), 65504)), codes
 *     clamp(rint(w * RN32(1 / d)), -127, 127) with the stored d (all zero when
 *     d is 0); a weight reads back as bf16(d * q);
 *   - adaLN modulation before a quantized linear: LayerNorm without affine
 *     terms over the features, times (1 + scale), plus shift, in binary64,
 *     rounded once to bf16; the W8A8 activation quantization then runs on
 *     that bf16 tensor unchanged;
 *   - GGUF Q4_K (same passage; the paper's encoder is its own and is not
 *     spelled out): round to nearest on a min-max grid per sub-block of 32,
 *     6-bit sub-block scales and offsets against binary16 super-block scales
 *     (256 weights), 4-bit codes against the stored grid; a weight reads
 *     back as bf16(RN32(d*sc*q - dmin*m)).
 *
 * Parallelism: rows are independent and each row is computed by one thread in
 * a fixed order, so results do not depend on the thread count.
 *
 * Build: gcc -O2 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_TINY_ABSMAX 0x1p-96f /* rows below this quantize to zero */

/* ------------------------------------------------------------------ */
/* bf16 <-> binary32 / binary64                                         */
/* ------------------------------------------------------------------ */

/* bf16 is the upper half of a binary32 word: widening is exact. */
static float bf16_to_float(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Round a finite binary64 value to the nearest bf16 (ties to even), in a
 * single rounding: bf16 keeps 8 significant bits and the binary32 exponent
 * range, with subnormals spaced 2^-133. */
static uint16_t double_to_bf16(double d)
{
    const double bf16_max = 0x1.fep127; /* (2 - 2^-7) * 2^127 */
    uint32_t u;
    float f;
    int e;
    int ulp_exp;
    double q;
    double r;

    if (d == 0.0)
        return signbit(d) ? 0x8000u : 0x0000u;
    frexp(fabs(d), &e);   /* |d| = m * 2^e with m in [0.5, 1) */
    ulp_exp = e - 8;      /* spacing of 8-significant-bit numbers there */
    if (ulp_exp < -133)
        ulp_exp = -133;   /* subnormal bf16 spacing */
    q = nearbyint(ldexp(d, -ulp_exp)); /* exact scaling, ties to even */
    r = ldexp(q, ulp_exp);
    if (fabs(r) > bf16_max)
        return signbit(d) ? 0xff80u : 0x7f80u; /* rounds to infinity */
    f = (float)r; /* exact: r has at most 8 significant bits */
    memcpy(&u, &f, sizeof u);
    return (uint16_t)(u >> 16);
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Exported so that the tests can pin the conversions on their own. */
float oracle_bf16_to_float(uint16_t h) { return bf16_to_float(h); }
uint16_t oracle_double_to_bf16(double d) { return double_to_bf16(d); }

/* ------------------------------------------------------------------ */
/* Calibration (Section 3, "INT8 W8A8": the per-channel activation      */
/* scales are measured beforehand over calibration inputs): the         */
/* per-input-channel absmax over tokens, and lambda.                    */
/* ------------------------------------------------------------------ */

/* s[k] = max(s[k], max_t |X[t][k]|). X is [M][K] bf16. The caller seeds s
 * (zeros for a fresh pass); several calls accumulate over batches. */
void oracle_act_absmax(const uint16_t *X, int64_t M, int64_t K, float *s)
{
    int64_t t, k;
    for (t = 0; t < M; ++t)
        for (k = 0; k < K; ++k) {
            float a = fabsf(bf16_to_float(X[t * K + k]));
            if (a > s[k])
                s[k] = a;
        }
}

/* lambda_j = s_j^alpha / (max_i |W_ij|)^(1 - alpha), W is [N][K] bf16 in the
 * nn.Linear layout (row i = output channel, column j = input channel). */
void oracle_smooth_factors(const float *act_absmax, const uint16_t *W,
                           int64_t N, int64_t K, double alpha, float *lambda)
{
    int64_t n, j;
    for (j = 0; j < K; ++j) {
        double wmax = 0.0;
        double s = (double)act_absmax[j];
        for (n = 0; n < N; ++n) {
            double a = fabs((double)bf16_to_float(W[n * K + j]));
            if (a > wmax)
                wmax = a;
        }
        if (s == 0.0 || wmax == 0.0) {
            lambda[j] = 1.0f;
            continue;
        }
        if (alpha == 0.5)
            lambda[j] = (float)(sqrt(s) / sqrt(wmax));
        else
            lambda[j] = (float)(pow(s, alpha) / pow(wmax, 1.0 - alpha));
    }
}

/* ------------------------------------------------------------------ */
/* Smoothing and symmetric per-row INT8 quantization.                  */
/* ------------------------------------------------------------------ */

/* One row: v_k = float(src_k) * mul_k (the smoothed row, one binary32
 * rounding), absmax over the row, scale = absmax/127, codes
 * clamp(rint(v_k * RN(127/absmax)), -127, 127). Two passes over the row, the
 * smoothed value recomputed in the second (it is the same binary32 number). */
static void smooth_quantize_row(const uint16_t *src, const float *mul,
                                int64_t K, int8_t *q, float *scale)
{
    int64_t k;
    float amax = 0.0f;
    float r;
    for (k = 0; k < K; ++k) {
        float a = fabsf(bf16_to_float(src[k]) * mul[k]);
        if (a > amax)
            amax = a;
    }
    if (amax < ORACLE_TINY_ABSMAX) {
        *scale = 0.0f;
        memset(q, 0, (size_t)K);
        return;
    }
    *scale = amax / 127.0f;
    r = 127.0f / amax;
    for (k = 0; k < K; ++k) {
        float v = bf16_to_float(src[k]) * mul[k];
        float c = rintf(v * r);
        if (c > 127.0f)
            c = 127.0f;
        if (c < -127.0f)
            c = -127.0f;
        q[k] = (int8_t)c;
    }
}

/* Offline weight preparation: W' = W * diag(lambda) (weights scaled up),
 * per-output-row INT8. W [N][K] bf16, lambda [K] -> Wq [N][K] int8,
 * w_scale [N], inv_lambda [K] (the activation-side multiplier). */
void oracle_prepare_weight(const uint16_t *W, const float *lambda, int64_t N,
                           int64_t K, int8_t *Wq, float *w_scale,
                           float *inv_lambda)
{
    int64_t n, k;
    for (k = 0; k < K; ++k)
        inv_lambda[k] = 1.0f / lambda[k];
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n)
        smooth_quantize_row(W + n * K, lambda, K, Wq + n * K, &w_scale[n]);
}

/* Runtime activation path: X' = X * diag(inv_lambda) (activations scaled
 * down), per-token INT8. X [M][K] bf16 -> Xq [M][K] int8, x_scale [M]. */
void oracle_quant_act(const uint16_t *X, const float *inv_lambda, int64_t M,
                      int64_t K, int8_t *Xq, float *x_scale)
{
    int64_t t;
#pragma omp parallel for schedule(static)
    for (t = 0; t < M; ++t)
        smooth_quantize_row(X + t * K, inv_lambda, K, Xq + t * K, &x_scale[t]);
}

/* adaLN modulation of a DiT block's input (the runtime-generated
 * modulation that Section 2 names as the reason smoothing is applied at
 * run time): h = LayerNorm(x) * (1 + scale) + shift per token, the norm over
 * the K features with no affine terms, then rounded once to bf16, the dtype
 * the model runs in. In binary64, in this order:
 *   mean = sum_k x_k / K,  var = sum_k (x_k - mean)^2 / K  (two passes),
 *   rstd = 1 / sqrt(var + eps),
 *   h_k = bf16(((x_k - mean) * rstd) * (1 + scale_k) + shift_k).
 * X [M][K], shift [K], scale [K] bf16 -> H [M][K] bf16. */
void oracle_adaln_modulate(const uint16_t *X, const uint16_t *shift, const uint16_t *scale,
                           int64_t M, int64_t K, double eps, uint16_t *H)
{
    int64_t t;
#pragma omp parallel for schedule(static)
    for (t = 0; t < M; ++t) {
        const uint16_t *x = X + t * K;
        double sum = 0.0, ss = 0.0, mean, rstd;
        int64_t k;
        for (k = 0; k < K; ++k)
            sum += (double)bf16_to_float(x[k]);
        mean = sum / (double)K;
        for (k = 0; k < K; ++k) {
            const double c = (double)bf16_to_float(x[k]) - mean;
            ss += c * c;
        }
        rstd = 1.0 / sqrt(ss / (double)K + eps);
        for (k = 0; k < K; ++k) {
            const double n = ((double)bf16_to_float(x[k]) - mean) * rstd;
            const double m = n * (1.0 + (double)bf16_to_float(scale[k]));
            H[t * K + k] = double_to_bf16(m + (double)bf16_to_float(shift[k]));
        }
    }
}

/* ------------------------------------------------------------------ */
/* INT8 GEMM and epilogue.                                              */
/* ------------------------------------------------------------------ */

/* C[t][n] = sum_k Xq[t][k] * Wq[n][k], exact in int32 (|C| <= 127^2 K, which
 * fits for K <= 133144). */
void oracle_gemm_i32(const int8_t *Xq, const int8_t *Wq, int64_t M, int64_t N,
                     int64_t K, int32_t *C)
{
    int64_t t, n, k;
#pragma omp parallel for schedule(static) private(n, k)
    for (t = 0; t < M; ++t)
        for (n = 0; n < N; ++n) {
            int32_t acc = 0;
            for (k = 0; k < K; ++k)
                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];
            C[t * N + n] = acc;
        }
}

/* Y[t][n] = bf16(C[t][n] * (s_tok[t] * s_ch[n]) + bias[n]), in binary64 with
 * one final rounding. bias may be NULL (treated as zero). */
void oracle_epilogue(const int32_t *C, const float *x_scale,
                     const float *w_scale, const uint16_t *bias, int64_t M,
                     int64_t N, uint16_t *Y)
{
    int64_t t, n;
#pragma omp parallel for schedule(static) private(n)
    for (t = 0; t < M; ++t)
        for (n = 0; n < N; ++n) {
            double b = bias ? (double)bf16_to_float(bias[n]) : 0.0;
            double y = (double)C[t * N + n] *
                           ((double)x_scale[t] * (double)w_scale[n]) + b;
            Y[t * N + n] = double_to_bf16(y);
        }
}

/* The W8A8 linear on already-quantized operands: the int32 sum and the
 * epilogue, row by row (no int32 matrix kept). */
void oracle_w8a8_linear(const int8_t *Xq, const float *x_scale,
                        const int8_t *Wq, const float *w_scale,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y)
{
    int64_t t, n, k;
#pragma omp parallel for schedule(static) private(n, k)
    for (t = 0; t < M; ++t)
        for (n = 0; n < N; ++n) {
            int32_t acc = 0;
            double b = bias ? (double)bf16_to_float(bias[n]) : 0.0;
            double y;
            for (k = 0; k < K; ++k)
                acc += (int32_t)Xq[t * K + k] * (int32_t)Wq[n * K + k];
            y = (double)acc * ((double)x_scale[t] * (double)w_scale[n]) + b;
            Y[t * N + n] = double_to_bf16(y);
        }
}

/* Protected layer: Y = bf16(X W^T + bias) with X, W bf16. The bf16 products
 * are exact in binary64; they are summed in binary64 in k order, the bias is
 * added last and the result is rounded once. bias may be NULL. */
void oracle_bf16_linear(const uint16_t *X, const uint16_t *W,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K,
                        uint16_t *Y)
{
    int64_t t, n, k;
#pragma omp parallel for schedule(static) private(n, k)
    for (t = 0; t < M; ++t)
        for (n = 0; n < N; ++n) {
            double acc = 0.0;
            for (k = 0; k < K; ++k)
                acc += (double)bf16_to_float(X[t * K + k]) *
                       (double)bf16_to_float(W[n * K + k]);
            if (bias)
                acc += (double)bf16_to_float(bias[n]);
            Y[t * N + n] = double_to_bf16(acc);
        }
}

/* ------------------------------------------------------------------ */
/* Fragility profile (Section 3, "Activation-fragility profiling and    */
/* protection"): per layer and denoising step, max |x|, standard        */
/* deviation and kurtosis of the linear's input activations.            */
/* ------------------------------------------------------------------ */

/* X is [M][K] bf16, n = M*K entries, mean = (1/n) sum x and
 * m_j = (1/n) sum (x - mean)^j. out[0] = max |x|, out[1] = mean,
 * out[2] = sqrt(m2) (population standard deviation), out[3] = m4 / m2^2
 * (Pearson kurtosis: 3 for a Gaussian), 0 when m2 = 0. Two passes in
 * binary64: the mean first, then the central sums. Each row's sums are
 * formed by one thread in k order and added in row order, so the result does
 * not depend on the thread count. Returns 0, or -1 if out of memory. */
int oracle_act_moments(const uint16_t *X, int64_t M, int64_t K, double *out)
{
    double *r1 = (double *)malloc((size_t)(M > 0 ? M : 1) * sizeof(double));
    double *r2 = (double *)malloc((size_t)(M > 0 ? M : 1) * sizeof(double));
    double *r4 = (double *)malloc((size_t)(M > 0 ? M : 1) * sizeof(double));
    float *rmax = (float *)malloc((size_t)(M > 0 ? M : 1) * sizeof(float));
    int64_t t, k;
    double n = (double)M * (double)K, s1 = 0.0, s2 = 0.0, s4 = 0.0, mean, m2, m4;
    float amax = 0.0f;
    if (!r1 || !r2 || !r4 || !rmax) {
        free(r1); free(r2); free(r4); free(rmax);
        return -1;
    }
#pragma omp parallel for schedule(static) private(k)
    for (t = 0; t < M; ++t) {
        double a = 0.0;
        float m = 0.0f;
        for (k = 0; k < K; ++k) {
            float x = bf16_to_float(X[t * K + k]);
            a += (double)x;
            if (fabsf(x) > m)
                m = fabsf(x);
        }
        r1[t] = a;
        rmax[t] = m;
    }
    for (t = 0; t < M; ++t) {
        s1 += r1[t];
        if (rmax[t] > amax)
            amax = rmax[t];
    }
    mean = s1 / n;
#pragma omp parallel for schedule(static) private(k)
    for (t = 0; t < M; ++t) {
        double a2 = 0.0, a4 = 0.0;
        for (k = 0; k < K; ++k) {
            double d = (double)bf16_to_float(X[t * K + k]) - mean;
            double d2 = d * d;
            a2 += d2;
            a4 += d2 * d2;
        }
        r2[t] = a2;
        r4[t] = a4;
    }
    for (t = 0; t < M; ++t) {
        s2 += r2[t];
        s4 += r4[t];
    }
    m2 = s2 / n;
    m4 = s4 / n;
    out[0] = (double)amax;
    out[1] = mean;
    out[2] = sqrt(m2);
    out[3] = m2 > 0.0 ? m4 / (m2 * m2) : 0.0;
    free(r1); free(r2); free(r4); free(rmax);
    return 0;
}

/* ------------------------------------------------------------------ */
/* GGUF Q8_0 weight-only format (Section 3, "GGUF k-quants": 8.5 bits    */
/* per weight, round to nearest).                                       */
/* ------------------------------------------------------------------ */

#define ORACLE_Q8_0_BLOCK 32
#define ORACLE_HALF_MAX 65504.0f

/* binary16 (1 sign, 5 exponent, 10 fraction bits) <-> binary32. */
static float half_to_float(uint16_t h)
{
    int e = (h >> 10) & 0x1f;
    double m = (double)(h & 0x3ff);
    double v;
    if (e == 0)
        v = ldexp(m, -24);                       /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m == 0.0 ? INFINITY : NAN;
    else
        v = ldexp(1024.0 + m, e - 25);           /* (1 + m/1024) * 2^(e-15) */
    return (float)((h & 0x8000) ? -v : v);
}

/* Round a finite binary32 value to the nearest binary16, ties to even, in a
 * single rounding (11 significant bits, subnormals spaced 2^-24). Values
 * that round past 65504 give infinity. */
static uint16_t float_to_half(float f)
{
    double d = (double)f, q, r;
    int e, ulp_exp;
    uint16_t sign = signbit(d) ? 0x8000u : 0u;
    if (d == 0.0)
        return sign;
    frexp(fabs(d), &e);                          /* |d| = m * 2^e, m in [0.5, 1) */
    ulp_exp = e - 11;
    if (ulp_exp < -24)
        ulp_exp = -24;
    q = nearbyint(ldexp(fabs(d), -ulp_exp));     /* exact scaling, ties to even */
    r = ldexp(q, ulp_exp);
    if (r > 65504.0)
        return sign | 0x7c00u;
    if (r < 0x1p-14)                             /* subnormal (or rounds to 2^-14) */
        return sign | (uint16_t)ldexp(r, 24);
    frexp(r, &e);                                /* r = m * 2^e */
    return sign | (uint16_t)(((e + 14) << 10) | ((uint32_t)ldexp(r, 11 - e) & 0x3ff));
}

uint16_t oracle_float_to_half(float f) { return float_to_half(f); }
float oracle_half_to_float(uint16_t h) { return half_to_float(h); }

/* W [N][K] bf16 (K a multiple of 32) -> codes qs [N][K] int8 and one scale
 * d [N][K/32] binary16 per block of 32 consecutive weights of a row:
 *   amax = max |w| over the block, d = RN16(min(RN32(amax / 127), 65504)),
 *   q = clamp(rint(w * RN32(1 / float(d))), -127, 127), all q = 0 if d = 0.
 * Binary32, one rounding per operation. */
void oracle_q8_0_quantize(const uint16_t *W, int64_t N, int64_t K, int8_t *qs,
                          uint16_t *d)
{
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        int64_t b;
        for (b = 0; b < K / ORACLE_Q8_0_BLOCK; ++b) {
            const uint16_t *w = W + n * K + b * ORACLE_Q8_0_BLOCK;
            int8_t *q = qs + n * K + b * ORACLE_Q8_0_BLOCK;
            float amax = 0.0f, s, inv, ds;
            int j;
            for (j = 0; j < ORACLE_Q8_0_BLOCK; ++j)
                if (fabsf(bf16_to_float(w[j])) > amax)
                    amax = fabsf(bf16_to_float(w[j]));
            s = amax / 127.0f;
            if (s > ORACLE_HALF_MAX)
                s = ORACLE_HALF_MAX;
            d[n * (K / ORACLE_Q8_0_BLOCK) + b] = float_to_half(s);
            ds = half_to_float(d[n * (K / ORACLE_Q8_0_BLOCK) + b]);
            inv = ds != 0.0f ? 1.0f / ds : 0.0f;
            for (j = 0; j < ORACLE_Q8_0_BLOCK; ++j) {
                float c = rintf(bf16_to_float(w[j]) * inv);
                if (c > 127.0f)
                    c = 127.0f;
                if (c < -127.0f)
                    c = -127.0f;
                q[j] = (int8_t)c;
            }
        }
    }
}

/* W'[n][k] = bf16(float(d[n][k / 32]) * qs[n][k]) (the product is exact in
 * binary32: 11 x 8 significant bits; one rounding to bf16). */
void oracle_q8_0_dequantize(const int8_t *qs, const uint16_t *d, int64_t N, int64_t K,
                            uint16_t *W)
{
    int64_t n, k;
#pragma omp parallel for schedule(static) private(k)
    for (n = 0; n < N; ++n)
        for (k = 0; k < K; ++k) {
            float v = half_to_float(d[n * (K / ORACLE_Q8_0_BLOCK) + k / ORACLE_Q8_0_BLOCK]) *
                      (float)qs[n * K + k];
            W[n * K + k] = double_to_bf16((double)v);
        }
}

/* ------------------------------------------------------------------ */
/* GGUF Q4_K weight-only format (Section 3, "GGUF k-quants": 4-bit      */
/* codes in super-blocks, the paper's own super-block quantizer).        */
/* A super-block is 256 consecutive weights of a row, cut into 8         */
/* sub-blocks of 32. A sub-block j reads back as                          */
/*   w = d * sc_j * q - dmin * m_j,  q in [0, 15], sc_j and m_j in [0, 63] */
/* with d and dmin binary16 per super-block. Stored planar:               */
/*   qs [N][K/2] (k even in the low nibble), scales [N][K/256][12] (the   */
/*   eight 6-bit sc_j and m_j of a super-block, packed below), d and dmin  */
/*   [N][K/256] binary16 bits: 4.5 bits per weight.                        */
/* ------------------------------------------------------------------ */

#define ORACLE_Q4_K_SUPER 256
#define ORACLE_Q4_K_SUB 32

static float cap_half(float v) { return v > ORACLE_HALF_MAX ? ORACLE_HALF_MAX : v; }

/* Round-to-nearest quantizer of one super-block, in three steps (binary32,
 * one rounding per operation):
 *   1. each sub-block's range: lo = min(0, min w), hi = max w,
 *      a_j = (hi - lo) / 15 (the step that spans it with 16 codes), b_j = -lo;
 *   2. the super-block scales: d = RN16(min(max_j a_j / 63, 65504)),
 *      dmin = RN16(min(max_j b_j / 63, 65504)); then the 6-bit sub-block
 *      scales sc_j = min(rint(a_j * RN32(1/d)), 63), m_j = min(rint(b_j * RN32(1/dmin)), 63)
 *      against the stored d and dmin (0 where d or dmin is 0);
 *   3. the codes against the stored grid: with s_j = d * sc_j and
 *      o_j = dmin * m_j (both exact), q = clamp(rint((w + o_j) * RN32(1/s_j)), 0, 15),
 *      q = 0 where s_j = 0. */
static void q4_k_super_block(const uint16_t *w, uint8_t *codes, uint8_t *sc, uint8_t *mn,
                             uint16_t *d, uint16_t *dmin)
{
    float a[8], b[8], amax = 0.0f, bmax = 0.0f, fd, fdm, inv_d, inv_dm;
    int j, i;
    for (j = 0; j < 8; ++j) {
        float lo = 0.0f, hi = -INFINITY;
        for (i = 0; i < ORACLE_Q4_K_SUB; ++i) {
            float v = bf16_to_float(w[j * ORACLE_Q4_K_SUB + i]);
            if (v < lo)
                lo = v;
            if (v > hi)
                hi = v;
        }
        a[j] = (hi - lo) / 15.0f;
        b[j] = -lo;
        if (a[j] > amax)
            amax = a[j];
        if (b[j] > bmax)
            bmax = b[j];
    }
    *d = float_to_half(cap_half(amax / 63.0f));
    *dmin = float_to_half(cap_half(bmax / 63.0f));
    fd = half_to_float(*d);
    fdm = half_to_float(*dmin);
    inv_d = fd != 0.0f ? 1.0f / fd : 0.0f;
    inv_dm = fdm != 0.0f ? 1.0f / fdm : 0.0f;
    for (j = 0; j < 8; ++j) {
        float cs = rintf(a[j] * inv_d), cm = rintf(b[j] * inv_dm), s, o, inv;
        if (cs > 63.0f)
            cs = 63.0f;
        if (cm > 63.0f)
            cm = 63.0f;
        sc[j] = (uint8_t)cs;
        mn[j] = (uint8_t)cm;
        s = fd * cs;
        o = fdm * cm;
        inv = s != 0.0f ? 1.0f / s : 0.0f;
        for (i = 0; i < ORACLE_Q4_K_SUB; ++i) {
            float c = rintf((bf16_to_float(w[j * ORACLE_Q4_K_SUB + i]) + o) * inv);
            if (c > 15.0f)
                c = 15.0f;
            if (c < 0.0f)
                c = 0.0f;
            codes[j * ORACLE_Q4_K_SUB + i] = (uint8_t)c;
        }
    }
}

/* The 8 sub-blocks' 6-bit scales sc_j and offsets m_j of a super-block in
 * 12 bytes, the GGUF k-quant scale layout (so that a super-block takes
 * 4 + (96 + 32) / 256 = 4.5 bits per weight): for j < 4, byte j holds sc_j
 * and byte j + 4 holds m_j in their low 6 bits; for j >= 4, byte j + 4
 * holds the low 4 bits of sc_j (low nibble) and of m_j (high nibble), and
 * their top 2 bits go to the top 2 bits of bytes j - 4 (sc_j) and j (m_j). */
void oracle_q4_k_pack_scales(const uint8_t *sc, const uint8_t *mn, uint8_t *out)
{
    int j;
    for (j = 0; j < 12; ++j)
        out[j] = 0;
    for (j = 0; j < 4; ++j) {
        out[j] |= (uint8_t)(sc[j] & 63);
        out[j + 4] |= (uint8_t)(mn[j] & 63);
    }
    for (j = 4; j < 8; ++j) {
        out[j + 4] = (uint8_t)((sc[j] & 15) | ((mn[j] & 15) << 4));
        out[j - 4] |= (uint8_t)((sc[j] >> 4) << 6);
        out[j] |= (uint8_t)((mn[j] >> 4) << 6);
    }
}

void oracle_q4_k_unpack_scales(const uint8_t *in, uint8_t *sc, uint8_t *mn)
{
    int j;
    for (j = 0; j < 4; ++j) {
        sc[j] = (uint8_t)(in[j] & 63);
        mn[j] = (uint8_t)(in[j + 4] & 63);
    }
    for (j = 4; j < 8; ++j) {
        sc[j] = (uint8_t)((in[j + 4] & 15) | ((in[j - 4] >> 6) << 4));
        mn[j] = (uint8_t)((in[j + 4] >> 4) | ((in[j] >> 6) << 4));
    }
}

/* W [N][K] bf16 (K a multiple of 256) -> qs [N][K/2], scales [N][K/256][12]
 * (packed as above), d, dmin [N][K/256]. */
void oracle_q4_k_quantize(const uint16_t *W, int64_t N, int64_t K, uint8_t *qs,
                          uint8_t *scales, uint16_t *d, uint16_t *dmin)
{
    int64_t n;
#pragma omp parallel for schedule(static)
    for (n = 0; n < N; ++n) {
        int64_t sb, k;
        uint8_t codes[ORACLE_Q4_K_SUPER], sc[8], mn[8];
        for (sb = 0; sb < K / ORACLE_Q4_K_SUPER; ++sb) {
            const int64_t sup = n * (K / ORACLE_Q4_K_SUPER) + sb;
            q4_k_super_block(W + n * K + sb * ORACLE_Q4_K_SUPER, codes, sc, mn, d + sup,
                             dmin + sup);
            oracle_q4_k_pack_scales(sc, mn, scales + 12 * sup);
            for (k = 0; k < ORACLE_Q4_K_SUPER; k += 2)
                qs[(n * K + sb * ORACLE_Q4_K_SUPER + k) / 2] =
                    (uint8_t)(codes[k] | (codes[k + 1] << 4));
        }
    }
}

/* W'[n][k] = bf16(RN32(d * sc_j * q - dmin * m_j)): d * sc_j * q (at most
 * 11 + 6 + 4 significant bits) and dmin * m_j are exact in binary32, their
 * difference is rounded once to binary32, then to bf16. */
void oracle_q4_k_dequantize(const uint8_t *qs, const uint8_t *scales, const uint16_t *d,
                            const uint16_t *dmin, int64_t N, int64_t K, uint16_t *W)
{
    int64_t n, k;
#pragma omp parallel for schedule(static) private(k)
    for (n = 0; n < N; ++n)
        for (k = 0; k < K; ++k) {
            const int64_t t = n * (K / ORACLE_Q4_K_SUPER) + k / ORACLE_Q4_K_SUPER;
            const int j = (int)((k % ORACLE_Q4_K_SUPER) / ORACLE_Q4_K_SUB);
            uint8_t sc[8], mn[8];
            const uint8_t byte = qs[(n * K + k) / 2];
            const float q = (float)((k & 1) ? byte >> 4 : byte & 15);
            float s, o, v;
            oracle_q4_k_unpack_scales(scales + 12 * t, sc, mn);
            s = half_to_float(d[t]) * (float)sc[j];
            o = half_to_float(dmin[t]) * (float)mn[j];
            v = s * q - o;
            W[n * K + k] = double_to_bf16((double)v);
        }
}
