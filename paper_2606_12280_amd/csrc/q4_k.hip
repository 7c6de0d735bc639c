// GGUF Q4_K weight-only format (paper Section 3, "GGUF k-quants": 4-bit
// codes in super-blocks, quantized by the paper's own super-block encoder).
// A super-block is 256 consecutive weights of a row, cut into 8 sub-blocks
// of 32; sub-block j reads back as
//   w = d * sc_j * q - dmin * m_j,   q in [0, 15], sc_j and m_j in [0, 63],
// with binary16 d and dmin per super-block. Round to nearest on a min-max
// grid, in binary32 with one rounding per operation:
//   1. per sub-block: lo = min(0, min w), hi = max w, a_j = (hi - lo) / 15,
//      b_j = -lo;
//   2. d = RN16(min(max_j a_j / 63, 65504)), dmin likewise from the b_j;
//      sc_j = min(rint(a_j * RN32(1/d)), 63), m_j = min(rint(b_j * RN32(1/dmin)), 63)
//      against the stored d and dmin (0 where they are 0);
//   3. s_j = d * sc_j and o_j = dmin * m_j (exact),
//      q = clamp(rint((w + o_j) * RN32(1/s_j)), 0, 15)   (0 where s_j = 0).
// A weight reads back as bf16(RN32(s_j * q - o_j)) (s_j * q is exact).
// Stored planar: qs [N][K/2] (even k in the low nibble), scales
// [N][K/256][12] (a super-block's eight 6-bit sc_j and m_j in the GGUF
// k-quant scale layout: for j < 4 bytes j and j + 4 hold sc_j and m_j in
// their low 6 bits; for j >= 4 byte j + 4 holds the low nibbles of sc_j and
// m_j, and their top two bits sit at the top of bytes j - 4 and j), d and
// dmin [N][K/256] binary16: 4 + (96 + 32) / 256 = 4.5 bits per weight.
//
// Dequantize is an HBM-bound stream: per weight 1/2 byte of codes and 1/16
// byte of scales in, 2 bytes of bf16 out.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace w8a8 {
namespace {

// The wave's index in its workgroup, in a scalar register.
__device__ __forceinline__ int wave_index() {
    return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
}

// The thread's unit under grid_for().
__device__ __forceinline__ int64_t unit_index() {
    return (static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x) * 256 + threadIdx.x;
}

constexpr int kSub = 32;
constexpr int kSubs = 8;  // sub-blocks per super-block
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    // one v_cvt_pk_bf16_f32 (round to nearest even), a in the low half
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

__device__ __forceinline__ float half_bits_to_float(uint16_t h) {
    return static_cast<float>(__builtin_bit_cast(_Float16, h));
}

__device__ __forceinline__ uint16_t float_to_half_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));  // round to nearest even
}

// The larger of a and b, keeping a unless b is strictly larger (so that a
// +0 start is never replaced by -0).
__device__ __forceinline__ float keep_max(float a, float b) { return b > a ? b : a; }

__device__ __forceinline__ float group8_max(float v) {
#pragma unroll
    for (int m = 1; m < kSubs; m <<= 1) v = keep_max(v, __shfl_xor(v, m, 64));
    return v;
}

__device__ __forceinline__ uint32_t group8_or(uint32_t v) {
#pragma unroll
    for (int m = 1; m < kSubs; m <<= 1) v |= __shfl_xor(v, m, 64);
    return v;
}

// One thread per sub-block; the 8 threads of a super-block are 8
// consecutive lanes, agree on d and dmin through lane shuffles, and OR
// their 6-bit values into the super-block's 12 scale bytes.
__global__ __launch_bounds__(256) void q4_k_quantize_kernel(
    const uint16_t *__restrict__ W, int64_t subs, uint8_t *__restrict__ qs,
    uint32_t *__restrict__ scales, uint16_t *__restrict__ d, uint16_t *__restrict__ dmin) {
    const int64_t j = unit_index();
    // subs is a multiple of 8 and groups of 8 lanes are aligned, so a
    // super-block's lanes are either all in range or all out.
    if (j >= subs) return;
    const uint4 *src = reinterpret_cast<const uint4 *>(W + j * kSub);
    float v[kSub];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const uint4 x = src[c];
        const uint32_t words[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[8 * c + 2 * e] = bf16_lo(words[e]);
            v[8 * c + 2 * e + 1] = bf16_hi(words[e]);
        }
    }
    float lo = 0.0f, hi = -__builtin_inff();
#pragma unroll
    for (int i = 0; i < kSub; ++i) {
        lo = v[i] < lo ? v[i] : lo;
        hi = v[i] > hi ? v[i] : hi;
    }
    const float a = (hi - lo) / 15.0f;
    const float b = -lo;
    const float amax = group8_max(keep_max(0.0f, a));
    const float bmax = group8_max(keep_max(0.0f, b));
    const uint16_t hd = float_to_half_bits(fminf(amax / 63.0f, 65504.0f));
    const uint16_t hdm = float_to_half_bits(fminf(bmax / 63.0f, 65504.0f));
    if ((j & (kSubs - 1)) == 0) {
        d[j / kSubs] = hd;
        dmin[j / kSubs] = hdm;
    }
    const float fd = half_bits_to_float(hd), fdm = half_bits_to_float(hdm);
    const float inv_d = fd != 0.0f ? 1.0f / fd : 0.0f;
    const float inv_dm = fdm != 0.0f ? 1.0f / fdm : 0.0f;
    const float cs = fminf(rintf(a * inv_d), 63.0f);
    const float cm = fminf(rintf(b * inv_dm), 63.0f);
    {
        const uint32_t vs = static_cast<uint32_t>(cs), vm = static_cast<uint32_t>(cm);
        const int jj = static_cast<int>(j & (kSubs - 1));
        const int sh = 8 * (jj & 3);
        uint32_t w0, w1, w2 = 0u;  // scale bytes 0-3, 4-7, 8-11
        if (jj < 4) {
            w0 = vs << sh;
            w1 = vm << sh;
        } else {
            w0 = (vs >> 4) << (sh + 6);
            w1 = (vm >> 4) << (sh + 6);
            w2 = ((vs & 15u) | ((vm & 15u) << 4)) << sh;
        }
        w0 = group8_or(w0);
        w1 = group8_or(w1);
        w2 = group8_or(w2);
        if (jj == 0) {
            uint32_t *o = scales + 3 * (j / kSubs);
            o[0] = w0;
            o[1] = w1;
            o[2] = w2;
        }
    }
    const float s = fd * cs, o = fdm * cm;
    const float inv = s != 0.0f ? 1.0f / s : 0.0f;
    uint32_t packed[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < kSub; ++i) {
        const float c = fminf(fmaxf(rintf((v[i] + o) * inv), 0.0f), 15.0f);
        packed[i / 8] |= static_cast<uint32_t>(c) << (4 * (i % 8));
    }
    reinterpret_cast<uint4 *>(qs)[j] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
}

// One thread per 8 weights: 4 bytes of codes and two binary16 scales in, 16
// bytes of bf16 out, so a wave's stores cover 1 KiB contiguously. A wave's
// 64 octets are exactly two super-blocks (its first octet is a multiple of
// 64), so the 12 scale bytes of both are wave-uniform: scalar loads, and
// each half of the wave takes its own. That leaves three vector loads per
// thread instead of six (36.1 -> 33.4 us at 16384 x 4096 in one job, output
// identical). The second super-block is clamped to the last one, so a wave
// whose upper half lies past the end reads nothing outside the planes.
__global__ __launch_bounds__(256) void q4_k_dequantize_kernel(
    const uint32_t *__restrict__ qs, const uint32_t *__restrict__ scales,
    const uint16_t *__restrict__ d, const uint16_t *__restrict__ dmin, int64_t octets,
    u32x4 *__restrict__ W) {
    const int lane = threadIdx.x & 63;
    const int wave = wave_index();
    const int64_t t0 =
        (static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x) * 256 + wave * 64;
    if (t0 >= octets) return;
    const int64_t supers = octets >> 5;  // 32 octets per super-block
    const int64_t g0 = t0 >> 5;
    const int64_t g1 = g0 + 1 < supers ? g0 + 1 : g0;
    const uint32_t a0 = scales[3 * g0], a1 = scales[3 * g0 + 1], a2 = scales[3 * g0 + 2];
    const uint32_t b0 = scales[3 * g1], b1 = scales[3 * g1 + 1], b2 = scales[3 * g1 + 2];
    const bool upper = lane >= 32;
    const uint32_t w0 = upper ? b0 : a0, w1 = upper ? b1 : a1, w2 = upper ? b2 : a2;
    const int64_t t = t0 + lane;
    if (t >= octets) return;
    const int64_t g = t >> 5;
    const int jj = static_cast<int>((t >> 2) & (kSubs - 1));  // sub-block in its super-block
    const uint32_t q = __builtin_nontemporal_load(qs + t);
    const uint16_t dh = d[g], mh = dmin[g];
    // the sub-block's 6-bit scale and offset, for both halves of the layout,
    // then the one for jj (a select, so both halves of a wave agree on the
    // path)
    const int sh = 8 * (jj & 3);
    const uint32_t lo = (w2 >> sh) & 255u;
    const uint32_t vs = jj < 4 ? (w0 >> sh) & 63u : (lo & 15u) | (((w0 >> (sh + 6)) & 3u) << 4);
    const uint32_t vm = jj < 4 ? (w1 >> sh) & 63u : (lo >> 4) | (((w1 >> (sh + 6)) & 3u) << 4);
    const float s = half_bits_to_float(dh) * static_cast<float>(vs);
    const float o = half_bits_to_float(mh) * static_cast<float>(vm);
    uint32_t out[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float q0 = static_cast<float>((q >> (8 * e)) & 15u);
        const float q1 = static_cast<float>((q >> (8 * e + 4)) & 15u);
        out[e] = bf16_pair(s * q0 - o, s * q1 - o);
    }
    __builtin_nontemporal_store(u32x4{out[0], out[1], out[2], out[3]}, W + t);
}

// Blocks of 256 threads for n units as a 2-D grid whose x extent stays at
// most 2^20 blocks, so that no dimension reaches 2^32 work-items.
dim3 grid_for(int64_t n) {
    const int64_t b = n > 0 ? (n + 255) / 256 : 1;
    const int64_t x = b < (INT64_C(1) << 20) ? b : (INT64_C(1) << 20);
    return dim3(static_cast<unsigned>(x), static_cast<unsigned>((b + x - 1) / x));
}

}  // namespace

hipError_t launch_q4_k_quantize(const uint16_t *W, int64_t N, int64_t K, uint8_t *qs,
                                uint8_t *scales, uint16_t *d, uint16_t *dmin,
                                hipStream_t stream) {
    const int64_t subs = N * (K / kSub);
    hipLaunchKernelGGL(q4_k_quantize_kernel, grid_for(subs), dim3(256), 0, stream, W, subs,
                       qs, reinterpret_cast<uint32_t *>(scales), d, dmin);
    return hipGetLastError();
}

hipError_t launch_q4_k_dequantize(const uint8_t *qs, const uint8_t *scales, const uint16_t *d,
                                  const uint16_t *dmin, int64_t N, int64_t K, uint16_t *W,
                                  hipStream_t stream) {
    const int64_t octets = N * K / 8;
    hipLaunchKernelGGL(q4_k_dequantize_kernel, grid_for(octets), dim3(256), 0, stream,
                       reinterpret_cast<const uint32_t *>(qs),
                       reinterpret_cast<const uint32_t *>(scales), d, dmin, octets,
                       reinterpret_cast<u32x4 *>(W));
    return hipGetLastError();
}

}  // namespace w8a8
