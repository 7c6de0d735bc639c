// adaLN modulation fused into the W8A8 activation quantization. In a DiT the
// input of the QKV and FFN-up projections is LayerNorm(x) * (1 + scale) +
// shift with a modulation generated at run time from the conditioning (the
// reason, given in paper Section 2, that smoothing cannot be folded into a
// preceding norm offline). This kernel computes, per token row,
//   mean = sum_k x_k / K,  var = sum_k (x_k - mean)^2 / K,
//   rstd = 1 / sqrt(var + eps),
//   h_k = bf16(((x_k - mean) * rstd) * (1 + scale_k) + shift_k)
// in binary64 (h is the bf16 tensor the unfused model would hold; the
// squares accumulate and the modulation applies with fused multiply-adds,
// which moves a binary64 result by at most an ulp of it), then the
// W8A8 activation step on h exactly as w8a8_quant_act does it: binary32
// v_k = float(h_k) * inv_lambda_k, absmax, scale absmax / 127, codes
// clamp(rint(v_k * RN(127 / absmax)), -127, 127). h never leaves registers:
// X is read once and the codes written once; run apart, the two steps would
// also write h and read it back (2 bytes each per element).
//
// Work mapping as in the quant kernel: a group of G waves owns a row, each
// lane CH chunks of 8 columns (consecutive lanes on consecutive 16-byte
// chunks), with its 8*CH smoothing multipliers and modulation values (as
// binary64) kept in registers across the RPW rows it walks; with RPW > 1 the
// next row is prefetched. The three row reductions (sum, centered sum of
// squares, absmax) run as lane butterflies, then across the G waves through
// LDS. The binary64 arithmetic (half the binary32 rate) bounds the kernel,
// not its bytes.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"
#include "wave_reduce.h"

namespace w8a8 {
namespace {

constexpr float kTinyAbsmax = 0x1p-96f;  // rows below quantize to zero

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
    const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ void store_stream(uint2 *p, uint32_t lo, uint32_t hi) {
    const v2u v = {lo, hi};
    __builtin_nontemporal_store(v, reinterpret_cast<v2u *>(p));
}

// The 8 bf16 values of a chunk, widened (exactly).
__device__ __forceinline__ void widen8(const uint4 &x, float (&v)[8]) {
    v[0] = bf16_lo(x.x);
    v[1] = bf16_hi(x.x);
    v[2] = bf16_lo(x.y);
    v[3] = bf16_hi(x.y);
    v[4] = bf16_lo(x.z);
    v[5] = bf16_hi(x.z);
    v[6] = bf16_lo(x.w);
    v[7] = bf16_hi(x.w);
}

// bf16 bits of a binary32 value, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    // one v_cvt_pk_bf16_f32 (round to nearest even), a in the low half
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// Nearest bf16 to a finite binary64 value in one rounding, given f, its
// nearest binary32: rounding f to bf16 gives the same result unless f lies
// exactly halfway between two bf16 values (low 16 bits 0x8000) while d does
// not; then d is on one side of that midpoint and decides. (binary32 refines
// the bf16 grid, subnormals included, so no other case differs.)
__device__ __forceinline__ bool bf16_midpoint(float f) {
    return (__float_as_uint(f) << 16) == 0x80000000u;
}

__device__ __forceinline__ uint32_t bf16_bits_past_midpoint(double d, float f) {
    const uint32_t t = __float_as_uint(f) >> 16;  // truncated toward zero
    if (static_cast<double>(f) == d) return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
    return fabs(d) > fabs(static_cast<double>(f)) ? t + 1 : t;
}

__device__ __forceinline__ double wave_sum(double v) { return lanes::sum(v); }
__device__ __forceinline__ float wave_max(float v) { return lanes::max(v); }

__device__ __forceinline__ uint32_t code(float v, float r) {
    float c = rintf(v * r);
    c = fminf(fmaxf(c, -127.0f), 127.0f);
    return static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xffu;
}

template <int G, int CH, int RPW, int WPB>
__global__ __launch_bounds__(WPB * 64) void adaln_quant_rows_kernel(
    const uint16_t *__restrict__ src, const uint16_t *__restrict__ shift,
    const uint16_t *__restrict__ scale, const float *__restrict__ mul, int64_t R, int64_t K,
    double eps, int8_t *__restrict__ out, float *__restrict__ xscale) {
    constexpr int SLOTS = WPB / G;
    static_assert(SLOTS * G == WPB, "G must divide WPB");
    __shared__ double red_sum[SLOTS][G];
    __shared__ double red_sq[SLOTS][G];
    __shared__ float red_max[SLOTS][G];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int sub = wave / G;
    const int gw = wave % G;
    const int64_t nchunk = K >> 3;
    const int64_t group = static_cast<int64_t>(blockIdx.x) * SLOTS + sub;
    const int64_t groups = static_cast<int64_t>(gridDim.x) * SLOTS;

    int64_t col[CH];
    bool live[CH];
    float4 ma[CH], mb[CH];
    double one_sc[CH][8], shd[CH][8];  // 1 + scale_k and shift_k, binary64
    const float4 *m4 = reinterpret_cast<const float4 *>(mul);
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        col[c] = static_cast<int64_t>(c) * (G * 64) + gw * 64 + lane;
        live[c] = col[c] < nchunk;
        const uint4 z = make_uint4(0u, 0u, 0u, 0u);
        ma[c] = live[c] ? m4[2 * col[c]] : make_float4(0.f, 0.f, 0.f, 0.f);
        mb[c] = live[c] ? m4[2 * col[c] + 1] : make_float4(0.f, 0.f, 0.f, 0.f);
        float fs[8], fh[8];
        widen8(live[c] ? reinterpret_cast<const uint4 *>(scale)[col[c]] : z, fs);
        widen8(live[c] ? reinterpret_cast<const uint4 *>(shift)[col[c]] : z, fh);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            one_sc[c][e] = 1.0 + static_cast<double>(fs[e]);
            shd[c][e] = static_cast<double>(fh[e]);
        }
    }

    uint4 x[CH];
    {
        const bool ok = group < R;
        const uint4 *srow = reinterpret_cast<const uint4 *>(src + (ok ? group : 0) * K);
#pragma unroll
        for (int c = 0; c < CH; ++c)
            x[c] = (ok && live[c]) ? load_stream(srow + col[c]) : make_uint4(0u, 0u, 0u, 0u);
    }
    for (int it = 0; it < RPW; ++it) {
        const int64_t row = group + it * groups;
        uint4 xn[CH];
        if (it + 1 < RPW) {
            const int64_t nrow = row + groups;
            const bool ok = nrow < R;
            const uint4 *srow = reinterpret_cast<const uint4 *>(src + (ok ? nrow : 0) * K);
#pragma unroll
            for (int c = 0; c < CH; ++c)
                xn[c] = (ok && live[c]) ? load_stream(srow + col[c]) : make_uint4(0u, 0u, 0u, 0u);
        }

        // mean (columns past K hold zeros and add nothing)
        double s = 0.0;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float v[8];
            widen8(x[c], v);
#pragma unroll
            for (int e = 0; e < 8; ++e) s += static_cast<double>(v[e]);
        }
        s = wave_sum(s);
        if constexpr (G > 1) {
            if (lane == 0) red_sum[sub][gw] = s;
            __syncthreads();
            s = red_sum[sub][0];
#pragma unroll
            for (int i = 1; i < G; ++i) s += red_sum[sub][i];
        }
        const double mean = s / static_cast<double>(K);

        // centered sum of squares (only live columns)
        double q = 0.0;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            if (!live[c]) continue;
            float v[8];
            widen8(x[c], v);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double d = static_cast<double>(v[e]) - mean;
                q = __builtin_fma(d, d, q);
            }
        }
        q = wave_sum(q);
        if constexpr (G > 1) {
            if (lane == 0) red_sq[sub][gw] = q;
            __syncthreads();
            q = red_sq[sub][0];
#pragma unroll
            for (int i = 1; i < G; ++i) q += red_sq[sub][i];
        }
        const double rstd = 1.0 / sqrt(q / static_cast<double>(K) + eps);

        // modulate, round to bf16 (kept packed in x), smoothed absmax
        float amax = 0.0f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float v[8], f[8];
            widen8(x[c], v);
            bool mid = false;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double n = (static_cast<double>(v[e]) - mean) * rstd;
                const double t = __builtin_fma(n, one_sc[c][e], shd[c][e]);
                f[e] = static_cast<float>(t);
                mid |= bf16_midpoint(f[e]);
            }
            uint32_t w[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) w[p] = bf16_pair(f[2 * p], f[2 * p + 1]);
            if (mid) {  // rare: a binary32 value on a bf16 midpoint
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    if (!bf16_midpoint(f[e])) continue;
                    const double n = (static_cast<double>(v[e]) - mean) * rstd;
                    const double t = __builtin_fma(n, one_sc[c][e], shd[c][e]);
                    const uint32_t h = bf16_bits_past_midpoint(t, f[e]);
                    const int sh = 16 * (e & 1);
                    w[e >> 1] = (w[e >> 1] & ~(0xffffu << sh)) | (h << sh);
                }
            }
            x[c] = make_uint4(w[0], w[1], w[2], w[3]);
            if (live[c]) {
                const float mv[8] = {ma[c].x, ma[c].y, ma[c].z, ma[c].w,
                                     mb[c].x, mb[c].y, mb[c].z, mb[c].w};
                float h[8];
                widen8(x[c], h);
#pragma unroll
                for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(h[e] * mv[e]));
            }
        }
        amax = wave_max(amax);
        if constexpr (G > 1) {
            if (lane == 0) red_max[sub][gw] = amax;
            __syncthreads();
#pragma unroll
            for (int i = 0; i < G; ++i) amax = fmaxf(amax, red_max[sub][i]);
        }

        if (row < R) {
            float scl = 0.0f;
            float r = 0.0f;
            const bool nonzero = amax >= kTinyAbsmax;
            if (nonzero) {
                scl = amax / 127.0f;
                r = 127.0f / amax;
            }
            if (gw == 0 && lane == 0) xscale[row] = scl;
            uint2 *orow = reinterpret_cast<uint2 *>(out + row * K);
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (!live[c]) continue;
                uint32_t lo = 0u;
                uint32_t hi = 0u;
                if (nonzero) {
                    float h[8];
                    widen8(x[c], h);
                    lo = code(h[0] * ma[c].x, r) | code(h[1] * ma[c].y, r) << 8 |
                         code(h[2] * ma[c].z, r) << 16 | code(h[3] * ma[c].w, r) << 24;
                    hi = code(h[4] * mb[c].x, r) | code(h[5] * mb[c].y, r) << 8 |
                         code(h[6] * mb[c].z, r) << 16 | code(h[7] * mb[c].w, r) << 24;
                }
                store_stream(orow + col[c], lo, hi);
            }
        }
        if (it + 1 < RPW) {
#pragma unroll
            for (int c = 0; c < CH; ++c) x[c] = xn[c];
        }
    }
}

template <int G, int CH, int RPW, int WPB>
hipError_t launch(const uint16_t *src, const uint16_t *shift, const uint16_t *scale,
                  const float *mul, int64_t R, int64_t K, double eps, int8_t *out,
                  float *xscale, hipStream_t stream) {
    constexpr int SLOTS = WPB / G;
    const int64_t groups = (R + RPW - 1) / RPW;
    const int64_t blocks = (groups + SLOTS - 1) / SLOTS;
    hipLaunchKernelGGL((adaln_quant_rows_kernel<G, CH, RPW, WPB>),
                       dim3(static_cast<unsigned>(blocks)), dim3(WPB * 64), 0, stream, src, shift,
                       scale, mul, R, K, eps, out, xscale);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_adaln_quant_act(const uint16_t *X, const uint16_t *shift,
                                  const uint16_t *scale, const float *inv_lambda, int64_t M,
                                  int64_t K, double eps, int8_t *Xq, float *x_scale,
                                  hipStream_t stream) {
    // A group covers G * 64 * CH * 8 columns; K <= 8192 (checked by the API:
    // a group of 8 waves with 4 chunks per lane would need more than the 256
    // registers two waves per SIMD may hold).
    if (K <= 512) return launch<1, 1, 2, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    if (K <= 1024) return launch<2, 1, 2, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    if (K <= 2048) return launch<4, 1, 2, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    // At K = 4096 a group walks two rows, loading the second while it works
    // on the first (4608 x 4096: 25.7 against 29.3 us for one row per group,
    // in one job; three rows per group measured the same as two).
    if (K <= 4096) return launch<4, 2, 2, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    return launch<8, 2, 1, 8>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
}

}  // namespace w8a8
