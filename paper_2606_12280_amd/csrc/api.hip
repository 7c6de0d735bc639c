// C ABI of libw8a8 (declared in include/w8a8.h): argument validation, then
// one or more kernel launches on the caller's stream. Validation touches no
// HIP state, so every error path can be exercised without a GPU.
#include "../../include/w8a8.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "internal.h"

namespace {

constexpr int kAbiVersion = 2;
constexpr int64_t kMaxRows = 1LL << 22;      // M (and N of the row kernels): grid size
constexpr int64_t kMaxN = 1LL << 20;         // GEMM output channels: 32-bit store offsets
constexpr int64_t kMaxMN = 1LL << 38;        // GEMM tiles: work-items below 2^32
constexpr int64_t kMaxK = 65536;             // one row per workgroup; 127^2 K < 2^31

thread_local char g_last_hip_error[160] = "";

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Span {
    const void *p;
    int64_t bytes;
};

bool overlap(Span a, Span b) {
    if (a.p == nullptr || b.p == nullptr || a.bytes <= 0 || b.bytes <= 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p);
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(b.p);
    return a0 < b0 + static_cast<uintptr_t>(b.bytes) && b0 < a0 + static_cast<uintptr_t>(a.bytes);
}

// Every output against every input and against the other outputs.
w8a8_status check_alias(std::initializer_list<Span> outs, std::initializer_list<Span> ins) {
    for (auto o = outs.begin(); o != outs.end(); ++o) {
        for (const Span &i : ins)
            if (overlap(*o, i)) return W8A8_ERR_ALIAS;
        for (auto o2 = o + 1; o2 != outs.end(); ++o2)
            if (overlap(*o, *o2)) return W8A8_ERR_ALIAS;
    }
    return W8A8_OK;
}

w8a8_status check_k(int64_t K) {
    if (K < 1) return W8A8_ERR_SHAPE;
    if (K % 64 != 0 || K > kMaxK) return W8A8_ERR_UNSUPPORTED;
    return W8A8_OK;
}

// The row kernels give a row of K > 32768 a workgroup of 1024 threads; 2^22
// such rows (512 GB of bf16) would make a grid of 2^32 work-items.
w8a8_status check_row_grid(int64_t rows, int64_t K) {
    return K > 32768 && rows >= kMaxRows ? W8A8_ERR_SHAPE : W8A8_OK;
}

w8a8_status check_rows(int64_t R, int64_t max_rows) {
    return (R < 1 || R > max_rows) ? W8A8_ERR_SHAPE : W8A8_OK;
}

// Token counts may be 0: an empty batch is validated like any other and
// then enqueues nothing.
w8a8_status check_tokens(int64_t M) {
    return (M < 0 || M > kMaxRows) ? W8A8_ERR_SHAPE : W8A8_OK;
}

// A buffer sized by the token count may be NULL when that count is 0.
bool missing(const void *p, int64_t M) { return p == nullptr && M > 0; }

w8a8_status hip_status(hipError_t e) {
    if (e == hipSuccess) return W8A8_OK;
    snprintf(g_last_hip_error, sizeof g_last_hip_error, "%s", hipGetErrorName(e));
    return W8A8_ERR_HIP;
}

#define W8A8_TRY(expr)                         \
    do {                                       \
        const w8a8_status s_ = (expr);         \
        if (s_ != W8A8_OK) return s_;          \
    } while (0)

hipStream_t as_stream(w8a8_stream s) { return static_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

int w8a8_abi_version(void) { return kAbiVersion; }

const char *w8a8_status_string(int status) {
    switch (status) {
        case W8A8_OK: return "ok";
        case W8A8_ERR_NULL: return "a required pointer is NULL";
        case W8A8_ERR_SHAPE: return "a size is out of range";
        case W8A8_ERR_ALIGN: return "a pointer is not aligned as required";
        case W8A8_ERR_ALIAS: return "an output overlaps an input or another output";
        case W8A8_ERR_UNSUPPORTED: return "unsupported request (K % 64, K > 65536 or alpha)";
        case W8A8_ERR_HIP: return "the HIP runtime reported an error";
        default: return "unknown status";
    }
}

const char *w8a8_last_hip_error(void) { return g_last_hip_error; }

w8a8_status w8a8_act_absmax(const uint16_t *X, int64_t M, int64_t K, float *absmax,
                            w8a8_stream stream) {
    if (missing(X, M) || absmax == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_k(K));
    if (!aligned(X, 16) || !aligned(absmax, 4)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{absmax, 4 * K}}, {{X, 2 * M * K}}));
    if (M == 0) return W8A8_OK;  // the running maximum is unchanged
    return hip_status(w8a8::launch_col_absmax(X, M, K, absmax, as_stream(stream)));
}

w8a8_status w8a8_act_moments(const uint16_t *X, int64_t M, int64_t K, void *work,
                             double *stats, w8a8_stream stream) {
    static_assert(W8A8_MOMENTS_WORK_BYTES == 6 * w8a8::kMomentBlocks * 8,
                  "workspace size");
    if (X == nullptr || work == nullptr || stats == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(M, kMaxRows));
    W8A8_TRY(check_k(K));
    if (!aligned(X, 16) || !aligned(work, 8) || !aligned(stats, 8)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{work, W8A8_MOMENTS_WORK_BYTES}, {stats, 32}}, {{X, 2 * M * K}}));
    return hip_status(w8a8::launch_act_moments(X, M * K, static_cast<double *>(work), stats,
                                               as_stream(stream)));
}

w8a8_status w8a8_act_moments_noalloc(const uint16_t *X, int64_t M, int64_t K, double *stats,
                                     w8a8_stream stream) {
    if (X == nullptr || stats == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(M, kMaxRows));
    W8A8_TRY(check_k(K));
    if (!aligned(X, 16) || !aligned(stats, 8)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{stats, 32}}, {{X, 2 * M * K}}));
    return hip_status(w8a8::launch_act_moments_noalloc(X, M * K, stats, as_stream(stream)));
}

w8a8_status w8a8_smooth_factors(const float *act_absmax, const uint16_t *W, int64_t N,
                                int64_t K, double alpha, float *lambda, w8a8_stream stream) {
    if (act_absmax == nullptr || W == nullptr || lambda == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(N, kMaxRows));
    W8A8_TRY(check_k(K));
    if (!(alpha > 0.0 && alpha < 1.0)) return W8A8_ERR_UNSUPPORTED;
    if (!aligned(W, 16) || !aligned(act_absmax, 4) || !aligned(lambda, 4)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{lambda, 4 * K}}, {{act_absmax, 4 * K}, {W, 2 * N * K}}));
    const hipStream_t s = as_stream(stream);
    W8A8_TRY(hip_status(w8a8::launch_zero_f32(lambda, K, s)));
    W8A8_TRY(hip_status(w8a8::launch_col_absmax(W, N, K, lambda, s)));
    return hip_status(w8a8::launch_lambda_from_stats(act_absmax, lambda, K, alpha, s));
}

w8a8_status w8a8_prepare_weight(const uint16_t *W, const float *lambda, int64_t N, int64_t K,
                                int8_t *Wq, float *w_scale, float *inv_lambda,
                                w8a8_stream stream) {
    if (W == nullptr || lambda == nullptr || Wq == nullptr || w_scale == nullptr ||
        inv_lambda == nullptr)
        return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(N, kMaxRows));
    W8A8_TRY(check_k(K));
    W8A8_TRY(check_row_grid(N, K));
    if (!aligned(W, 16) || !aligned(Wq, 16) || !aligned(lambda, 16) || !aligned(w_scale, 4) ||
        !aligned(inv_lambda, 4))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{Wq, N * K}, {w_scale, 4 * N}, {inv_lambda, 4 * K}},
                         {{W, 2 * N * K}, {lambda, 4 * K}}));
    const hipStream_t s = as_stream(stream);
    W8A8_TRY(hip_status(w8a8::launch_reciprocal(lambda, K, inv_lambda, s)));
    return hip_status(w8a8::launch_smooth_quant_rows(W, lambda, N, K, Wq, w_scale, s));
}

w8a8_status w8a8_quant_act(const uint16_t *X, const float *inv_lambda, int64_t M, int64_t K,
                           int8_t *Xq, float *x_scale, w8a8_stream stream) {
    if (missing(X, M) || inv_lambda == nullptr || missing(Xq, M) || missing(x_scale, M))
        return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_k(K));
    W8A8_TRY(check_row_grid(M, K));
    if (!aligned(X, 16) || !aligned(Xq, 16) || !aligned(inv_lambda, 16) || !aligned(x_scale, 4))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{Xq, M * K}, {x_scale, 4 * M}}, {{X, 2 * M * K}, {inv_lambda, 4 * K}}));
    if (M == 0) return W8A8_OK;
    return hip_status(
        w8a8::launch_smooth_quant_rows(X, inv_lambda, M, K, Xq, x_scale, as_stream(stream)));
}

w8a8_status w8a8_adaln_quant_act(const uint16_t *X, const uint16_t *shift, const uint16_t *scale,
                                 const float *inv_lambda, int64_t M, int64_t K, double eps,
                                 int8_t *Xq, float *x_scale, w8a8_stream stream) {
    if (missing(X, M) || shift == nullptr || scale == nullptr || inv_lambda == nullptr ||
        missing(Xq, M) || missing(x_scale, M))
        return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_k(K));
    if (K > 8192 || !(eps >= 0.0) || !std::isfinite(eps)) return W8A8_ERR_UNSUPPORTED;
    if (!aligned(X, 16) || !aligned(shift, 16) || !aligned(scale, 16) || !aligned(Xq, 16) ||
        !aligned(inv_lambda, 16) || !aligned(x_scale, 4))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{Xq, M * K}, {x_scale, 4 * M}},
                         {{X, 2 * M * K}, {shift, 2 * K}, {scale, 2 * K}, {inv_lambda, 4 * K}}));
    if (M == 0) return W8A8_OK;
    return hip_status(w8a8::launch_adaln_quant_act(X, shift, scale, inv_lambda, M, K, eps, Xq,
                                                   x_scale, as_stream(stream)));
}

w8a8_status w8a8_linear(const int8_t *Xq, const float *x_scale, const int8_t *Wq,
                        const float *w_scale, const uint16_t *bias, int64_t M, int64_t N,
                        int64_t K, uint16_t *Y, w8a8_stream stream) {
    if (missing(Xq, M) || missing(x_scale, M) || Wq == nullptr || w_scale == nullptr ||
        missing(Y, M))
        return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    W8A8_TRY(check_k(K));
    if (!aligned(Xq, 16) || !aligned(Wq, 16) || !aligned(Y, 16) || !aligned(x_scale, 4) ||
        !aligned(w_scale, 4) || !aligned(bias, 2))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{Y, 2 * M * N}}, {{Xq, M * K},
                                            {x_scale, 4 * M},
                                            {Wq, N * K},
                                            {w_scale, 4 * N},
                                            {bias, bias ? 2 * N : 0}}));
    if (M == 0) return W8A8_OK;
    return hip_status(w8a8::launch_gemm_i8(Xq, Wq, x_scale, w_scale, bias, M, N, K, Y, nullptr,
                                           as_stream(stream)));
}

w8a8_status w8a8_gemm_i32(const int8_t *Xq, const int8_t *Wq, int64_t M, int64_t N, int64_t K,
                          int32_t *C, w8a8_stream stream) {
    if (missing(Xq, M) || Wq == nullptr || missing(C, M)) return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    W8A8_TRY(check_k(K));
    if (!aligned(Xq, 16) || !aligned(Wq, 16) || !aligned(C, 16)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{C, 4 * M * N}}, {{Xq, M * K}, {Wq, N * K}}));
    if (M == 0) return W8A8_OK;
    return hip_status(w8a8::launch_gemm_i8(Xq, Wq, nullptr, nullptr, nullptr, M, N, K, nullptr, C,
                                           as_stream(stream)));
}

w8a8_status bf16_linear(const uint16_t *X, const uint16_t *W, const uint16_t *bias, int64_t M,
                        int64_t N, int64_t K, uint16_t *Y, w8a8_stream stream) {
    if (missing(X, M) || W == nullptr || missing(Y, M)) return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    W8A8_TRY(check_k(K));
    if (!aligned(X, 16) || !aligned(W, 16) || !aligned(Y, 16) || !aligned(bias, 2))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{Y, 2 * M * N}},
                         {{X, 2 * M * K}, {W, 2 * N * K}, {bias, bias ? 2 * N : 0}}));
    if (M == 0) return W8A8_OK;
    return hip_status(w8a8::launch_gemm_bf16(X, W, bias, M, N, K, Y, as_stream(stream)));
}

w8a8_status w8a8_gemm_config(int64_t M, int64_t N, int64_t K, int bf16, int32_t *tile_m,
                             int32_t *tile_n, int32_t *threads) {
    if (tile_m == nullptr || tile_n == nullptr || threads == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(M, kMaxRows));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    W8A8_TRY(check_k(K));
    int bm = 0, bn = 0, nt = 0;
    w8a8::gemm_config(M, N, bf16 ? 2 * K : K, &bm, &bn, &nt);
    *tile_m = bm;
    *tile_n = bn;
    *threads = nt;
    return W8A8_OK;
}

w8a8_status q8_0_quantize(const uint16_t *W, int64_t N, int64_t K, int8_t *qs, uint16_t *d,
                          w8a8_stream stream) {
    if (W == nullptr || qs == nullptr || d == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(N, kMaxRows));
    W8A8_TRY(check_k(K));
    if (!aligned(W, 16) || !aligned(qs, 16) || !aligned(d, 2)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{qs, N * K}, {d, N * (K / 32) * 2}}, {{W, 2 * N * K}}));
    return hip_status(w8a8::launch_q8_0_quantize(W, N, K, qs, d, as_stream(stream)));
}

w8a8_status q8_0_dequantize(const int8_t *qs, const uint16_t *d, int64_t N, int64_t K,
                            uint16_t *W, w8a8_stream stream) {
    if (qs == nullptr || d == nullptr || W == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(N, kMaxRows));
    W8A8_TRY(check_k(K));
    if (!aligned(W, 16) || !aligned(qs, 16) || !aligned(d, 2)) return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{W, 2 * N * K}}, {{qs, N * K}, {d, N * (K / 32) * 2}}));
    return hip_status(w8a8::launch_q8_0_dequantize(qs, d, N, K, W, as_stream(stream)));
}

w8a8_status q8_0_linear(const uint16_t *X, const int8_t *qs, const uint16_t *d,
                        const uint16_t *bias, int64_t M, int64_t N, int64_t K, uint16_t *work,
                        uint16_t *Y, w8a8_stream stream) {
    if (missing(X, M) || qs == nullptr || d == nullptr || work == nullptr || missing(Y, M))
        return W8A8_ERR_NULL;
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    W8A8_TRY(check_k(K));
    if (!aligned(X, 16) || !aligned(qs, 16) || !aligned(d, 2) || !aligned(work, 16) ||
        !aligned(Y, 16) || !aligned(bias, 2))
        return W8A8_ERR_ALIGN;
    W8A8_TRY(check_alias({{work, 2 * N * K}, {Y, 2 * M * N}},
                         {{X, 2 * M * K}, {qs, N * K}, {d, N * (K / 32) * 2},
                          {bias, bias ? 2 * N : 0}}));
    if (M == 0) return W8A8_OK;
    const hipStream_t s = as_stream(stream);
    W8A8_TRY(hip_status(w8a8::launch_q8_0_dequantize(qs, d, N, K, work, s)));
    return hip_status(w8a8::launch_gemm_bf16(X, work, bias, M, N, K, Y, s));
}

// Q4_K plane sizes in bytes for W [N][K].
struct Q4kPlanes {
    int64_t qs, scales, super;
};
static Q4kPlanes q4_k_planes(int64_t N, int64_t K) {
    return {N * K / 2, 12 * N * (K / 256), 2 * N * (K / 256)};
}

static w8a8_status check_q4_k_args(const uint8_t *qs, const uint8_t *scales, const uint16_t *d,
                                   const uint16_t *dmin, int64_t N, int64_t K) {
    if (qs == nullptr || scales == nullptr || d == nullptr || dmin == nullptr)
        return W8A8_ERR_NULL;
    W8A8_TRY(check_rows(N, kMaxRows));
    W8A8_TRY(check_k(K));
    if (K % 256 != 0) return W8A8_ERR_UNSUPPORTED;
    if (!aligned(qs, 16) || !aligned(scales, 4) || !aligned(d, 2) || !aligned(dmin, 2))
        return W8A8_ERR_ALIGN;
    return W8A8_OK;
}

w8a8_status q4_k_quantize(const uint16_t *W, int64_t N, int64_t K, uint8_t *qs, uint8_t *scales,
                          uint16_t *d, uint16_t *dmin, w8a8_stream stream) {
    if (W == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_q4_k_args(qs, scales, d, dmin, N, K));
    if (!aligned(W, 16)) return W8A8_ERR_ALIGN;
    const Q4kPlanes b = q4_k_planes(N, K);
    W8A8_TRY(check_alias({{qs, b.qs}, {scales, b.scales}, {d, b.super}, {dmin, b.super}},
                         {{W, 2 * N * K}}));
    return hip_status(w8a8::launch_q4_k_quantize(W, N, K, qs, scales, d, dmin, as_stream(stream)));
}

w8a8_status q4_k_dequantize(const uint8_t *qs, const uint8_t *scales, const uint16_t *d,
                            const uint16_t *dmin, int64_t N, int64_t K, uint16_t *W,
                            w8a8_stream stream) {
    if (W == nullptr) return W8A8_ERR_NULL;
    W8A8_TRY(check_q4_k_args(qs, scales, d, dmin, N, K));
    if (!aligned(W, 16)) return W8A8_ERR_ALIGN;
    const Q4kPlanes b = q4_k_planes(N, K);
    W8A8_TRY(check_alias({{W, 2 * N * K}},
                         {{qs, b.qs}, {scales, b.scales}, {d, b.super}, {dmin, b.super}}));
    return hip_status(
        w8a8::launch_q4_k_dequantize(qs, scales, d, dmin, N, K, W, as_stream(stream)));
}

w8a8_status q4_k_linear(const uint16_t *X, const uint8_t *qs, const uint8_t *scales,
                        const uint16_t *d, const uint16_t *dmin, const uint16_t *bias, int64_t M,
                        int64_t N, int64_t K, uint16_t *work, uint16_t *Y, w8a8_stream stream) {
    if (missing(X, M) || work == nullptr || missing(Y, M)) return W8A8_ERR_NULL;
    W8A8_TRY(check_q4_k_args(qs, scales, d, dmin, N, K));
    W8A8_TRY(check_tokens(M));
    W8A8_TRY(check_rows(N, kMaxN));
    if (M * N > kMaxMN) return W8A8_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(work, 16) || !aligned(Y, 16) || !aligned(bias, 2))
        return W8A8_ERR_ALIGN;
    const Q4kPlanes b = q4_k_planes(N, K);
    W8A8_TRY(check_alias({{work, 2 * N * K}, {Y, 2 * M * N}},
                         {{X, 2 * M * K}, {qs, b.qs}, {scales, b.scales}, {d, b.super},
                          {dmin, b.super}, {bias, bias ? 2 * N : 0}}));
    if (M == 0) return W8A8_OK;
    const hipStream_t s = as_stream(stream);
    W8A8_TRY(hip_status(w8a8::launch_q4_k_dequantize(qs, scales, d, dmin, N, K, work, s)));
    return hip_status(w8a8::launch_gemm_bf16(X, work, bias, M, N, K, Y, s));
}

}  // extern "C"
