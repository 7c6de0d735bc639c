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
// Work mapping: a group of G waves owns a row, each lane CH chunks of 8
// columns (consecutive lanes on consecutive 16-byte chunks), with its 8*CH
// smoothing multipliers and modulation values (as binary64) kept in
// registers across the rows it walks. One launch holds as many groups as the
// GPU keeps resident, each walking an equal share of the rows with the next
// row prefetched. The three row reductions (sum, centered sum of squares,
// absmax) run as lane butterflies, then across the G waves through LDS. The
// vector ALU's issue bounds the kernel, not its bytes: about 27 VALU instructions
// per element of a lane, nearly a third of them binary64.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"
#include "row_io.h"
#include "wave_reduce.h"

namespace w8a8 {
namespace {

constexpr float kTinyAbsmax = 0x1p-96f;  // rows below quantize to zero

using rows::code_word;
using rows::load_chunk;
using rows::make_rsrc;
using rows::pack4;
using rows::store_codes;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

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
// v is a running absmax (fmaxf of fabsf values from 0), so never NaN or negative.
__device__ __forceinline__ float wave_max(float v) { return lanes::max_nonneg(v); }

template <int G, int CH, int WPB>
__global__ __launch_bounds__(WPB * 64) void adaln_quant_rows_kernel(
    const uint16_t *__restrict__ src, const uint16_t *__restrict__ shift,
    const uint16_t *__restrict__ scale, const float *__restrict__ mul, int64_t R, int64_t K,
    double eps, int rows_per_group, int8_t *__restrict__ out, float *__restrict__ xscale) {
    constexpr int SLOTS = WPB / G;
    static_assert(SLOTS * G == WPB, "G must divide WPB");
    __shared__ double red_sum[SLOTS][G];
    __shared__ double red_sq[SLOTS][G];
    __shared__ float red_max[SLOTS][G];
    const int lane = threadIdx.x & 63;
    // wave-uniform (in a scalar register), so that the row resources are too
    const int wave = rows::wave_index();
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
            // opaque: kept in registers across the rows rather than derived
            // again from the bf16 words for every row (three binary64
            // operations per element)
            asm volatile("" : "+v"(one_sc[c][e]), "+v"(shd[c][e]));
        }
    }
    // The two divisions by K: a multiplication by 1/K when K is a power of
    // two (exact, so the same bits as the division), else the division.
    const bool k_pow2 = (K & (K - 1)) == 0;
    const double inv_k = 1.0 / static_cast<double>(K);

    // the rows' resources: K bf16 in, K codes out, one scale out; empty past
    // the input
    const auto row_in = [&](int64_t r) {
        return make_rsrc(src + (r < R ? r : 0) * K, r < R ? static_cast<uint32_t>(K) * 2u : 0u);
    };
    uint32_t in_off[CH], out_off[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        in_off[c] = live[c] ? static_cast<uint32_t>(col[c]) * 16u : 0xfffffff0u;
        out_off[c] = live[c] ? static_cast<uint32_t>(col[c]) * 8u : 0xfffffff8u;
    }
    const uint32_t scale_off = (gw == 0 && lane == 0) ? 0u : 4u;

    // A row's scale and codes out (a row past the input stores nothing).
    const auto store_row = [&](int64_t r, float scl, const uint32_t (&lo)[CH],
                               const uint32_t (&hi)[CH]) {
        const bool in = r < R;
        rows::store_f32(make_rsrc(xscale + (in ? r : 0), in ? 4u : 0u), scale_off, scl);
        const __amdgpu_buffer_rsrc_t ro =
            make_rsrc(out + (in ? r : 0) * K, in ? static_cast<uint32_t>(K) : 0u);
#pragma unroll
        for (int c = 0; c < CH; ++c) store_codes(ro, out_off[c], lo[c], hi[c]);
    };

    uint4 x[CH];
    {
        const __amdgpu_buffer_rsrc_t rin = row_in(group);
#pragma unroll
        for (int c = 0; c < CH; ++c) x[c] = load_chunk(rin, in_off[c]);
    }
    // A row's scale and codes go out one row late, right after the next
    // row's sum exchange: the GPU counts vector loads and stores on one
    // counter, and the compiler's wait for a row's data also waits for every
    // store issued after that data's loads, so stores at the end of a row
    // would hold up the next row by a store's full latency. The first
    // pending row lies past the input, so its stores are dropped.
    uint32_t pend_lo[CH], pend_hi[CH];
    float pend_scl = 0.0f;
    int64_t pend_row = R;
#pragma unroll
    for (int c = 0; c < CH; ++c) pend_lo[c] = pend_hi[c] = 0u;
    for (int it = 0; it < rows_per_group; ++it) {
        const int64_t row = group + it * groups;
        // the next row (past the last row of the group it lies past the
        // input, so nothing is read)
        uint4 xn[CH];
        {
            const __amdgpu_buffer_rsrc_t rin = row_in(row + groups);
#pragma unroll
            for (int c = 0; c < CH; ++c) xn[c] = load_chunk(rin, in_off[c]);
        }

        // the row in binary64 (exact) and its sum; columns past K hold zeros
        // and add nothing
        // (two partial sums per lane, halving the dependent chain)
        double xd[CH][8];
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float v[8];
            widen8(x[c], v);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                xd[c][e] = static_cast<double>(v[e]);
                if (e & 1) s1 += xd[c][e];
                else s0 += xd[c][e];
            }
        }
        double s = wave_sum(s0 + s1);
        if constexpr (G > 1) {
            if (lane == 0) red_sum[sub][gw] = s;
            __syncthreads();
            s = red_sum[sub][0];
#pragma unroll
            for (int i = 1; i < G; ++i) s += red_sum[sub][i];
        }
        const double mean = k_pow2 ? s * inv_k : s / static_cast<double>(K);
        __builtin_amdgcn_sched_barrier(0);  // after this row's data was waited for
        store_row(pend_row, pend_scl, pend_lo, pend_hi);

        // centered values (kept for the modulation) and their sum of squares
        // (only live columns)
        double q0 = 0.0, q1 = 0.0;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            if (!live[c]) continue;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                xd[c][e] -= mean;
                if (e & 1) q1 = __builtin_fma(xd[c][e], xd[c][e], q1);
                else q0 = __builtin_fma(xd[c][e], xd[c][e], q0);
            }
        }
        double q = wave_sum(q0 + q1);
        if constexpr (G > 1) {
            if (lane == 0) red_sq[sub][gw] = q;
            __syncthreads();
            q = red_sq[sub][0];
#pragma unroll
            for (int i = 1; i < G; ++i) q += red_sq[sub][i];
        }
        const double var = k_pow2 ? q * inv_k : q / static_cast<double>(K);
        const double rstd = 1.0 / sqrt(var + eps);

        // modulate, round to bf16, smooth (kept in registers), absmax
        float hv[CH][8];
        float amax = 0.0f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            float f[8];
            bool mid = false;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double t = __builtin_fma(xd[c][e] * rstd, one_sc[c][e], shd[c][e]);
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
                    const double t = __builtin_fma(xd[c][e] * rstd, one_sc[c][e], shd[c][e]);
                    const uint32_t h = bf16_bits_past_midpoint(t, f[e]);
                    const int sh = 16 * (e & 1);
                    w[e >> 1] = (w[e >> 1] & ~(0xffffu << sh)) | (h << sh);
                }
            }
            float h[8];
            widen8(make_uint4(w[0], w[1], w[2], w[3]), h);
            const float mv[8] = {ma[c].x, ma[c].y, ma[c].z, ma[c].w,
                                 mb[c].x, mb[c].y, mb[c].z, mb[c].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) hv[c][e] = h[e] * mv[e];
            if (live[c]) {
#pragma unroll
                for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(hv[c][e]));
            }
        }
        amax = wave_max(amax);
        if constexpr (G > 1) {
            if (lane == 0) red_max[sub][gw] = amax;
            __syncthreads();
#pragma unroll
            for (int i = 0; i < G; ++i) amax = fmaxf(amax, red_max[sub][i]);
        }

        {
            float scl = 0.0f;
            float r = 0.0f;
            const bool nonzero = amax >= kTinyAbsmax;
            if (nonzero) {
                scl = amax / 127.0f;
                r = 127.0f / amax;
            }
            pend_row = row;
            pend_scl = scl;
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                pend_lo[c] = 0u;
                pend_hi[c] = 0u;
                if (nonzero) {
                    pend_lo[c] = pack4(code_word(hv[c][0], r), code_word(hv[c][1], r),
                                       code_word(hv[c][2], r), code_word(hv[c][3], r));
                    pend_hi[c] = pack4(code_word(hv[c][4], r), code_word(hv[c][5], r),
                                       code_word(hv[c][6], r), code_word(hv[c][7], r));
                }
            }
        }
#pragma unroll
        for (int c = 0; c < CH; ++c) x[c] = xn[c];
    }
    store_row(pend_row, pend_scl, pend_lo, pend_hi);
}

// One round of groups: as many as the GPU holds at once (fewer for short
// inputs), each walking rows_per_group rows, so that the per-column
// constants each group loads serve several rows and no second, partial
// round of groups is left at the end.
template <int G, int CH, int WPB>
hipError_t launch(const uint16_t *src, const uint16_t *shift, const uint16_t *scale,
                  const float *mul, int64_t R, int64_t K, double eps, int8_t *out,
                  float *xscale, hipStream_t stream) {
    constexpr int SLOTS = WPB / G;
    if (R <= 0) return hipSuccess;
    static std::atomic<int64_t> resident[256];
    const int64_t rpg = rows::rows_per_group(
        R, rows::resident_groups(
               reinterpret_cast<const void *>(&adaln_quant_rows_kernel<G, CH, WPB>), WPB * 64,
               SLOTS, resident));
    if (rpg > INT32_MAX) return hipErrorInvalidValue;
    const int64_t groups = (R + rpg - 1) / rpg;
    const int64_t blocks = (groups + SLOTS - 1) / SLOTS;
    hipLaunchKernelGGL((adaln_quant_rows_kernel<G, CH, WPB>), dim3(static_cast<unsigned>(blocks)),
                       dim3(WPB * 64), 0, stream, src, shift, scale, mul, R, K, eps,
                       static_cast<int>(rpg), out, xscale);
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
    if (K <= 512) return launch<1, 1, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    if (K <= 1024) return launch<2, 1, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    if (K <= 2048) return launch<4, 1, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    if (K <= 4096) return launch<4, 2, 4>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
    return launch<8, 2, 8>(X, shift, scale, inv_lambda, M, K, eps, Xq, x_scale, stream);
}

}  // namespace w8a8
