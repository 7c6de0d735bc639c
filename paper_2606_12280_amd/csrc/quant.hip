// Memory-bound kernels of the W8A8 recipe (paper Section 3, "INT8 W8A8"):
//   - smooth + per-row INT8 quantization (activations per token at run time,
//     weights per output channel offline);
//   - the reciprocal of the smoothing factors;
//   - calibration: per-channel absmax and the smoothing equation
//     lambda_j = s_j^alpha / max_i |W_ij|^(1-alpha).
//
// Row quantization: a group of G wavefronts owns one row. Each lane owns CH
// chunks of 8 columns (consecutive lanes on consecutive 16-byte chunks, so
// every wave load is one contiguous 1 KiB) and keeps the matching 8 smoothing
// multipliers of each chunk in registers for all the rows it visits. One
// launch holds as many groups as the GPU keeps resident, each walking an
// equal share of the rows and loading the next row while it reduces and
// writes the current one:
//   absmax over the row (lane shuffles, then across the G waves in LDS),
//   scale, then 8 codes per chunk as one 8-byte store.
// The smoothed value float(x) * mul is recomputed for the coding pass rather
// than held, which halves the registers a row needs; it is the same binary32
// product both times. X is read exactly once and the codes written once,
// both with nontemporal hints (streamed through the caches, not kept).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"
#include "row_io.h"
#include "wave_reduce.h"

namespace w8a8 {
namespace {

constexpr float kTinyAbsmax = 0x1p-96f;  // rows below quantize to zero

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// v is a running absmax (fmaxf of fabsf values from 0), so never NaN or negative.
__device__ __forceinline__ float wave_max(float v) { return lanes::max_nonneg(v); }

// The 8 smoothed values of one chunk: float(x_e) * mul_e, one binary32
// rounding each.
__device__ __forceinline__ void smooth8(const uint4 &x, const float4 &ma, const float4 &mb,
                                        float (&v)[8]) {
    v[0] = bf16_lo(x.x) * ma.x;
    v[1] = bf16_hi(x.x) * ma.y;
    v[2] = bf16_lo(x.y) * ma.z;
    v[3] = bf16_hi(x.y) * ma.w;
    v[4] = bf16_lo(x.z) * mb.x;
    v[5] = bf16_hi(x.z) * mb.y;
    v[6] = bf16_lo(x.w) * mb.z;
    v[7] = bf16_hi(x.w) * mb.w;
}

__device__ __forceinline__ float absmax8(const uint4 &x, const float4 &ma, const float4 &mb,
                                         float a) {
    float v[8];
    smooth8(x, ma, mb, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) a = fmaxf(a, fabsf(v[e]));
    return a;
}

// WPB waves per block hold WPB / G row groups. Every wave runs exactly
// rows_per_group iterations, so the LDS barrier is uniform; rows past R read
// zeros and store nothing. Group g of the grid visits rows g, g + groups,
// g + 2 groups, ... With PF the next row is loaded while the current one is
// reduced and coded. Without (the K = 65536 group has no register room for
// a second row) a group takes one row and the grid covers the rows.
template <int G, int CH, int WPB, bool PF>
__global__ __launch_bounds__(WPB * 64) void smooth_quant_rows_kernel(
    const uint16_t *__restrict__ src, const float *__restrict__ mul, int64_t R,
    int64_t K, int rows_per_group, int8_t *__restrict__ out, float *__restrict__ scale) {
    constexpr int SLOTS = WPB / G;
    static_assert(SLOTS * G == WPB, "G must divide WPB");
    __shared__ float red[2][SLOTS][G];
    const int lane = threadIdx.x & 63;
    const int wave = rows::wave_index();
    const int sub = wave / G;
    const int gw = wave % G;
    const int64_t nchunk = K >> 3;
    const int64_t group = static_cast<int64_t>(blockIdx.x) * SLOTS + sub;
    const int64_t groups = static_cast<int64_t>(gridDim.x) * SLOTS;

    // chunk c of the lane: col(c); a chunk past K has its byte offsets past
    // the row, so its loads read zeros and its stores are dropped
    const uint32_t col0 = static_cast<uint32_t>(gw * 64 + lane);
    const auto col = [&](int c) { return col0 + static_cast<uint32_t>(c * G * 64); };
    float4 ma[CH], mb[CH];
    const float4 *m4 = reinterpret_cast<const float4 *>(mul);
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const bool live = col(c) < nchunk;
        ma[c] = live ? m4[2 * col(c)] : make_float4(0.f, 0.f, 0.f, 0.f);
        mb[c] = live ? m4[2 * col(c) + 1] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const uint32_t scale_off = (gw == 0 && lane == 0) ? 0u : 4u;
    // the rows' resources: K bf16 in, K codes out, one scale out; empty past
    // the input
    const auto load_row = [&](int64_t r, uint4 (&x)[CH]) {
        const __amdgpu_buffer_rsrc_t rin =
            rows::make_rsrc(src + (r < R ? r : 0) * K, r < R ? static_cast<uint32_t>(K) * 2u : 0u);
#pragma unroll
        for (int c = 0; c < CH; ++c) x[c] = rows::load_chunk(rin, col(c) * 16u);
    };

    // A row's scale and codes out (a row past the input stores nothing).
    const auto store_row = [&](int64_t r, float sc, const uint32_t (&lo)[CH],
                               const uint32_t (&hi)[CH]) {
        const bool in = r < R;
        rows::store_f32(rows::make_rsrc(scale + (in ? r : 0), in ? 4u : 0u), scale_off, sc);
        const __amdgpu_buffer_rsrc_t ro =
            rows::make_rsrc(out + (in ? r : 0) * K, in ? static_cast<uint32_t>(K) : 0u);
#pragma unroll
        for (int c = 0; c < CH; ++c) rows::store_codes(ro, col(c) * 8u, lo[c], hi[c]);
    };

    uint4 x[CH];
    if constexpr (PF) load_row(group, x);
    const int n_rows = PF ? rows_per_group : 1;
    // With the prefetch, a row's scale and codes go out one row late, right
    // after the next row's absmax exchange. The GPU counts vector loads and
    // stores on one counter, and the compiler's wait for a row's data also
    // waits for every store issued after that data's loads: stores at the
    // end of a row would hold up the next row by a store's full latency.
    // The first pending row lies past the input, so its stores are dropped.
    uint32_t pend_lo[CH], pend_hi[CH];
    float pend_sc = 0.0f;
    int64_t pend_row = R;
#pragma unroll
    for (int c = 0; c < CH; ++c) pend_lo[c] = pend_hi[c] = 0u;
    for (int it = 0; it < n_rows; ++it) {
        const int64_t row = group + it * groups;
        uint4 xn[CH];
        // the next row (past the group's last row it lies past the input,
        // so nothing is read)
        if constexpr (PF) load_row(row + groups, xn);
        else load_row(row, x);
        float amax = 0.0f;
#pragma unroll
        for (int c = 0; c < CH; ++c) amax = absmax8(x[c], ma[c], mb[c], amax);
        amax = wave_max(amax);
        if constexpr (G > 1) {
            if (lane == 0) red[it & 1][sub][gw] = amax;
            __syncthreads();
#pragma unroll
            for (int i = 0; i < G; ++i) amax = fmaxf(amax, red[it & 1][sub][i]);
        }
        if constexpr (PF) {
            __builtin_amdgcn_sched_barrier(0);  // after this row's data was waited for
            store_row(pend_row, pend_sc, pend_lo, pend_hi);
        }
        float sc = 0.0f;
        float r = 0.0f;
        const bool nonzero = amax >= kTinyAbsmax;
        if (nonzero) {
            sc = amax / 127.0f;
            r = 127.0f / amax;
        }
        uint32_t lo[CH], hi[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            lo[c] = 0u;
            hi[c] = 0u;
            if (nonzero) {
                float t[8];
                smooth8(x[c], ma[c], mb[c], t);
                lo[c] = rows::pack4(rows::code_word(t[0], r), rows::code_word(t[1], r),
                                    rows::code_word(t[2], r), rows::code_word(t[3], r));
                hi[c] = rows::pack4(rows::code_word(t[4], r), rows::code_word(t[5], r),
                                    rows::code_word(t[6], r), rows::code_word(t[7], r));
            }
        }
        if constexpr (PF) {
            pend_row = row;
            pend_sc = sc;
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                pend_lo[c] = lo[c];
                pend_hi[c] = hi[c];
                x[c] = xn[c];
            }
        } else {
            store_row(row, sc, lo, hi);
        }
    }
    if constexpr (PF) store_row(pend_row, pend_sc, pend_lo, pend_hi);
}

// One round of groups: as many as the GPU holds at once (fewer for short
// inputs), each walking an equal share of the rows.
template <int G, int CH, int WPB, bool PF>
hipError_t launch_rows(const uint16_t *src, const float *mul, int64_t R, int64_t K,
                       int8_t *out, float *scale, hipStream_t stream) {
    constexpr int SLOTS = WPB / G;
    if (R <= 0) return hipSuccess;
    static std::atomic<int64_t> resident[256];
    const int64_t rpg =
        PF ? rows::rows_per_group(
                 R, rows::resident_groups(
                        reinterpret_cast<const void *>(&smooth_quant_rows_kernel<G, CH, WPB, PF>),
                        WPB * 64, SLOTS, resident))
           : 1;
    if (rpg > INT32_MAX) return hipErrorInvalidValue;
    const int64_t groups = (R + rpg - 1) / rpg;
    const int64_t blocks = (groups + SLOTS - 1) / SLOTS;
    // A grid of 2^32 work-items or more cannot be launched. Only one row per
    // group gets there: R = 2^22 rows with K > 32768, 512 GB of bf16, more
    // than the GPU holds.
    if (blocks * WPB * 64 >= (INT64_C(1) << 32)) return hipErrorInvalidValue;
    hipLaunchKernelGGL((smooth_quant_rows_kernel<G, CH, WPB, PF>),
                       dim3(static_cast<unsigned>(blocks)), dim3(WPB * 64), 0, stream, src, mul,
                       R, K, static_cast<int>(rpg), out, scale);
    return hipGetLastError();
}

__global__ void reciprocal_kernel(const float *__restrict__ lam, int64_t K,
                                  float *__restrict__ inv) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k < K) inv[k] = 1.0f / lam[k];
}

__global__ void zero_kernel(float *__restrict__ dst, int64_t K) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k < K) dst[k] = 0.0f;
}

// Column absmax: a workgroup covers 8 CPW columns (16 CPW bytes of every
// row) of a strip of rows. Lane l of wave w reads the 8 columns of chunk
// l % CPW in row (64 / CPW) w + l / CPW of every step of 16 (64 / CPW) rows,
// so each wave load is 64 / CPW row segments of 16 CPW bytes, with
// kColUnroll steps in flight. Lanes holding the same chunk combine with lane
// shuffles, the waves in LDS, and one integer atomic max per column leaves
// the workgroup (the bit patterns of non-negative floats order like the
// floats). Strips are sized for about kColTarget workgroups, so a column
// sees about kColTarget / (K / (8 CPW)) atomics: atomics on one address
// serialize at the memory side.
constexpr int64_t kColTarget = 512;
constexpr int kColWaves = 16;
constexpr int kColUnroll = 4;

template <int CPW>
__global__ __launch_bounds__(kColWaves * 64) void col_absmax_kernel(
    const uint16_t *__restrict__ src, int64_t R, int64_t K, int64_t strip,
    float *__restrict__ colmax) {
    static_assert(CPW >= 8 && CPW <= 64 && (CPW & (CPW - 1)) == 0, "chunks per segment");
    constexpr int RPL = 64 / CPW;              // rows per wave load
    constexpr int STEP = kColWaves * RPL;      // rows per workgroup step
    __shared__ float red[kColWaves][CPW][9];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int chunk = lane % CPW;
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * (8 * CPW) + chunk * 8;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * strip;
    const int64_t r1 = r0 + strip < R ? r0 + strip : R;
    float m[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int64_t r = r0 + wave * RPL + lane / CPW; r < r1; r += STEP * kColUnroll) {
        uint4 x[kColUnroll];
#pragma unroll
        for (int u = 0; u < kColUnroll; ++u) {
            const int64_t ru = r + STEP * u;
            x[u] = ru < r1 ? *reinterpret_cast<const uint4 *>(src + ru * K + c0)
                           : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < kColUnroll; ++u) {
            m[0] = fmaxf(m[0], fabsf(bf16_lo(x[u].x)));
            m[1] = fmaxf(m[1], fabsf(bf16_hi(x[u].x)));
            m[2] = fmaxf(m[2], fabsf(bf16_lo(x[u].y)));
            m[3] = fmaxf(m[3], fabsf(bf16_hi(x[u].y)));
            m[4] = fmaxf(m[4], fabsf(bf16_lo(x[u].z)));
            m[5] = fmaxf(m[5], fabsf(bf16_hi(x[u].z)));
            m[6] = fmaxf(m[6], fabsf(bf16_lo(x[u].w)));
            m[7] = fmaxf(m[7], fabsf(bf16_hi(x[u].w)));
        }
    }
    // lanes l, l ^ CPW, l ^ 2 CPW, ... hold the same chunk
#pragma unroll
    for (int d = CPW; d < 64; d <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = fmaxf(m[e], __shfl_xor(m[e], d, 64));
    if (lane < CPW) {
#pragma unroll
        for (int e = 0; e < 8; ++e) red[wave][lane][e] = m[e];
    }
    __syncthreads();
    for (int t = threadIdx.x; t < 8 * CPW; t += kColWaves * 64) {
        const int ch = t >> 3;
        const int e = t & 7;
        float v = red[0][ch][e];
        for (int w = 1; w < kColWaves; ++w) v = fmaxf(v, red[w][ch][e]);
        atomicMax(reinterpret_cast<unsigned int *>(colmax) + blockIdx.x * (8 * CPW) + t,
                  __float_as_uint(v));
    }
}

__global__ void lambda_kernel(const float *__restrict__ s, float *__restrict__ lam, int64_t K,
                              double alpha) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k >= K) return;
    const double sk = static_cast<double>(s[k]);
    const double wk = static_cast<double>(lam[k]);  // weight column absmax
    float out = 1.0f;
    if (sk != 0.0 && wk != 0.0) {
        if (alpha == 0.5)
            out = static_cast<float>(sqrt(sk) / sqrt(wk));
        else
            out = static_cast<float>(pow(sk, alpha) / pow(wk, 1.0 - alpha));
    }
    lam[k] = out;
}

unsigned blocks_for(int64_t n, int threads) {
    return static_cast<unsigned>((n + threads - 1) / threads);
}

}  // namespace

hipError_t launch_smooth_quant_rows(const uint16_t *src, const float *mul, int64_t R,
                                    int64_t K, int8_t *out, float *scale,
                                    hipStream_t stream) {
    // A group covers 512 * G * CH columns; take the smallest that holds K.
    if (K <= 512) return launch_rows<1, 1, 4, true>(src, mul, R, K, out, scale, stream);
    if (K <= 1024) return launch_rows<2, 1, 4, true>(src, mul, R, K, out, scale, stream);
    if (K <= 2048) return launch_rows<4, 1, 4, true>(src, mul, R, K, out, scale, stream);
    if (K <= 4096) return launch_rows<4, 2, 4, true>(src, mul, R, K, out, scale, stream);
    if (K <= 8192) return launch_rows<8, 2, 8, true>(src, mul, R, K, out, scale, stream);
    if (K <= 16384) return launch_rows<8, 4, 8, true>(src, mul, R, K, out, scale, stream);
    if (K <= 32768) return launch_rows<8, 8, 8, true>(src, mul, R, K, out, scale, stream);
    return launch_rows<16, 8, 16, false>(src, mul, R, K, out, scale, stream);  // K <= 65536
}

hipError_t launch_reciprocal(const float *lam, int64_t K, float *inv, hipStream_t stream) {
    hipLaunchKernelGGL(reciprocal_kernel, dim3(blocks_for(K, 256)), dim3(256), 0, stream, lam,
                       K, inv);
    return hipGetLastError();
}

hipError_t launch_zero_f32(float *dst, int64_t K, hipStream_t stream) {
    hipLaunchKernelGGL(zero_kernel, dim3(blocks_for(K, 256)), dim3(256), 0, stream, dst, K);
    return hipGetLastError();
}

template <int CPW>
hipError_t launch_col_absmax_cpw(const uint16_t *src, int64_t R, int64_t K, float *colmax,
                                 hipStream_t stream) {
    const int64_t gx = K / (8 * CPW);
    const int64_t step = kColWaves * (64 / CPW);
    int64_t strips = (kColTarget + gx - 1) / gx;
    const int64_t max_strips = (R + step - 1) / step;  // a step of rows at least
    if (strips > max_strips) strips = max_strips;
    if (strips < 1) strips = 1;
    const int64_t strip = (R + strips - 1) / strips;
    const dim3 grid(static_cast<unsigned>(gx), static_cast<unsigned>((R + strip - 1) / strip));
    hipLaunchKernelGGL(col_absmax_kernel<CPW>, grid, dim3(kColWaves * 64), 0, stream, src, R, K,
                       strip, colmax);
    return hipGetLastError();
}

hipError_t launch_col_absmax(const uint16_t *src, int64_t R, int64_t K, float *colmax,
                             hipStream_t stream) {
    // 512-byte row segments where K allows (4608 x 4096: 8.4 us against 9.9
    // for 128-byte and 8.4 for 1 KiB segments; 4608 x 16384: 25.7 against
    // 31.3 and 27.2 us; in one job). The entry point guarantees 64 | K.
    if (K % 256 == 0) return launch_col_absmax_cpw<32>(src, R, K, colmax, stream);
    if (K % 128 == 0) return launch_col_absmax_cpw<16>(src, R, K, colmax, stream);
    return launch_col_absmax_cpw<8>(src, R, K, colmax, stream);
}

hipError_t launch_lambda_from_stats(const float *s, float *lam, int64_t K, double alpha,
                                    hipStream_t stream) {
    hipLaunchKernelGGL(lambda_kernel, dim3(blocks_for(K, 256)), dim3(256), 0, stream, s, lam, K,
                       alpha);
    return hipGetLastError();
}

}  // namespace w8a8
