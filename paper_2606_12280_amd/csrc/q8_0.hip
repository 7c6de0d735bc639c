// GGUF Q8_0 weight-only format (paper Section 3, "GGUF k-quants": 8.5 bits
// per weight, round to nearest). A row of W [N][K] is cut into blocks of 32
// consecutive weights; a block keeps 32 int8 codes and one binary16 scale:
//   amax = max |w|, d = RN16(min(RN32(amax / 127), 65504)),
//   q = clamp(rint(w * RN32(1 / float(d))), -127, 127)   (all 0 if d == 0),
// and a weight reads back as bf16(float(d) * q) (the product is exact in
// binary32; one rounding). Codes and scales are stored planar: qs [N][K] int8
// and d [N][K/32] binary16, 8.5 bits per weight in all.
//
// Both kernels are HBM-bound streaming passes: quantize reads 2 bytes and
// writes 1 + 1/16 per weight; dequantize reads 1 + 1/16 and writes 2.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace w8a8 {
namespace {

// The thread's unit under grid_for().
__device__ __forceinline__ int64_t unit_index() {
    return (static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x) * 256 + threadIdx.x;
}

constexpr int kBlock = 32;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    // one v_cvt_pk_bf16_f32 (round to nearest even), a in the low half
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

__device__ __forceinline__ uint32_t code4(const float *v, float inv) {
    uint32_t r = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        float c = rintf(v[e] * inv);
        c = fminf(fmaxf(c, -127.0f), 127.0f);
        r |= (static_cast<uint32_t>(static_cast<int32_t>(c)) & 0xffu) << (8 * e);
    }
    return r;
}

// One thread per block of 32 weights (64 bytes of bf16 in, 34 bytes out).
__global__ __launch_bounds__(256) void q8_0_quantize_kernel(const uint16_t *__restrict__ W,
                                                            int64_t blocks,
                                                            int8_t *__restrict__ qs,
                                                            uint16_t *__restrict__ d) {
    const int64_t b = unit_index();
    if (b >= blocks) return;
    const uint4 *src = reinterpret_cast<const uint4 *>(W + b * kBlock);
    float v[kBlock];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const uint4 x = src[c];
        v[8 * c + 0] = bf16_lo(x.x);
        v[8 * c + 1] = bf16_hi(x.x);
        v[8 * c + 2] = bf16_lo(x.y);
        v[8 * c + 3] = bf16_hi(x.y);
        v[8 * c + 4] = bf16_lo(x.z);
        v[8 * c + 5] = bf16_hi(x.z);
        v[8 * c + 6] = bf16_lo(x.w);
        v[8 * c + 7] = bf16_hi(x.w);
    }
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < kBlock; ++j) amax = fmaxf(amax, fabsf(v[j]));
    const float s = fminf(amax / 127.0f, 65504.0f);
    const _Float16 h = static_cast<_Float16>(s);  // v_cvt_f16_f32: round to nearest even
    d[b] = __builtin_bit_cast(uint16_t, h);
    const float ds = static_cast<float>(h);
    const float inv = ds != 0.0f ? 1.0f / ds : 0.0f;
    uint4 *dst = reinterpret_cast<uint4 *>(qs + b * kBlock);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const float *t = v + 16 * c;
        dst[c] = make_uint4(code4(t, inv), code4(t + 4, inv), code4(t + 8, inv),
                            code4(t + 12, inv));
    }
}

// One thread per 8 codes: 8 bytes of codes and the block's scale in, 16
// bytes of bf16 out, so a wave's stores cover 1 KiB contiguously. Codes in
// and weights out carry nontemporal hints (streamed once).
__global__ __launch_bounds__(256) void q8_0_dequantize_kernel(const u32x2 *__restrict__ qs,
                                                              const uint16_t *__restrict__ d,
                                                              int64_t octets,
                                                              u32x4 *__restrict__ W) {
    const int64_t t = unit_index();
    if (t >= octets) return;
    const float ds = static_cast<float>(__builtin_bit_cast(_Float16, d[t >> 2]));
    const u32x2 q = __builtin_nontemporal_load(qs + t);
    uint32_t out[4];
#pragma unroll
    for (int w = 0; w < 2; ++w) {
        const int32_t v = static_cast<int32_t>(q[w]);
        const float c0 = static_cast<float>((v << 24) >> 24);
        const float c1 = static_cast<float>((v << 16) >> 24);
        const float c2 = static_cast<float>((v << 8) >> 24);
        const float c3 = static_cast<float>(v >> 24);
        out[2 * w] = bf16_pair(ds * c0, ds * c1);
        out[2 * w + 1] = bf16_pair(ds * c2, ds * c3);
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

hipError_t launch_q8_0_quantize(const uint16_t *W, int64_t N, int64_t K, int8_t *qs,
                                uint16_t *d, hipStream_t stream) {
    const int64_t blocks = N * (K / kBlock);
    hipLaunchKernelGGL(q8_0_quantize_kernel, grid_for(blocks), dim3(256), 0, stream, W,
                       blocks, qs, d);
    return hipGetLastError();
}

hipError_t launch_q8_0_dequantize(const int8_t *qs, const uint16_t *d, int64_t N, int64_t K,
                                  uint16_t *W, hipStream_t stream) {
    const int64_t octets = N * K / 8;
    hipLaunchKernelGGL(q8_0_dequantize_kernel, grid_for(octets), dim3(256), 0, stream,
                       reinterpret_cast<const u32x2 *>(qs), d, octets,
                       reinterpret_cast<u32x4 *>(W));
    return hipGetLastError();
}

}  // namespace w8a8
