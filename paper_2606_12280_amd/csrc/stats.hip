// Fragility profile of a linear's input (paper Section 3, "Activation-
// fragility profiling and protection"): max |x|, mean, population standard
// deviation and Pearson kurtosis m4 / m2^2 over all entries of X, in binary64.
//
// Two passes over X: the sum and max |x|, then the central sums of the second
// and fourth powers around the mean (the mean is never folded into raw power
// sums, which would cancel). Both passes use a fixed grid of kMomentBlocks
// workgroups walking X in 16-byte chunks with a fixed stride; each workgroup
// reduces in a fixed order and writes its partials to the caller's workspace,
// and a single workgroup adds those in order. Every call on the same input
// therefore returns the same bits. The passes are HBM-bound. The first pass
// reads X with ordinary loads, so that an X of up to ~200 MB (every DiT
// linear input) is still in the 256 MB last-level cache for the second,
// which reads it nontemporally. Each thread keeps 4 chunk loads in flight.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace w8a8 {
namespace {

constexpr int kThreads = 256;
constexpr int kFinalThreads = 1024;

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
    const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Sum over a workgroup of NT threads, in a fixed order: butterfly within each
// wave, then the wave totals in wave order by thread 0 (valid there only).
template <int NT>
__device__ __forceinline__ double group_sum(double v, double *red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    double t = 0.0;
    if (threadIdx.x == 0)
        for (int w = 0; w < NT / 64; ++w) t += red[w];
    __syncthreads();
    return t;
}

template <int NT>
__device__ __forceinline__ float group_max(float v, float *red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    float t = 0.0f;
    if (threadIdx.x == 0)
        for (int w = 0; w < NT / 64; ++w) t = fmaxf(t, red[w]);
    __syncthreads();
    return t;
}

constexpr int kUnroll = 4;  // chunk loads in flight per thread

// Chunks of thread `tid` of the grid: tid, tid + stride, ... in groups of
// kUnroll (loads first, then the arithmetic in chunk order). Chunks past
// the end read as zero and are skipped by `valid`.
template <bool STREAM, class F>
__device__ __forceinline__ void for_chunks(const uint4 *__restrict__ X, int64_t chunks, F &&f) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    for (int64_t c0 = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; c0 < chunks;
         c0 += kUnroll * stride) {
        uint4 x[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t c = c0 + u * stride;
            x[u] = c < chunks ? (STREAM ? load_stream(X + c) : X[c]) : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (c0 + u * stride < chunks) f(x[u]);
    }
}

// Pass 1: part[2 b] = sum of x, part[2 b + 1] = max |x| over workgroup b's chunks.
__global__ __launch_bounds__(kThreads) void moments_sum_kernel(const uint4 *__restrict__ X,
                                                               int64_t chunks,
                                                               double *__restrict__ part) {
    __shared__ double red[kThreads / 64];
    __shared__ float redf[kThreads / 64];
    double s = 0.0;
    float m = 0.0f;
    for_chunks<false>(X, chunks, [&](const uint4 &x) {
        const float v[8] = {lo(x.x), hi(x.x), lo(x.y), hi(x.y), lo(x.z), hi(x.z), lo(x.w), hi(x.w)};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            s += static_cast<double>(v[e]);
            m = fmaxf(m, fabsf(v[e]));
        }
    });
    s = group_sum<kThreads>(s, red);
    m = group_max<kThreads>(m, redf);
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = s;
        part[2 * blockIdx.x + 1] = static_cast<double>(m);
    }
}

// mm[0] = mean = (sum of the partial sums) / n, mm[1] = max |x|.
__global__ __launch_bounds__(kFinalThreads) void moments_mean_kernel(
    const double *__restrict__ part, int blocks, double n, double *__restrict__ mm) {
    __shared__ double red[kFinalThreads / 64];
    __shared__ float redf[kFinalThreads / 64];
    double s = 0.0;
    float m = 0.0f;
    for (int b = threadIdx.x; b < blocks; b += kFinalThreads) {
        s += part[2 * b];
        m = fmaxf(m, static_cast<float>(part[2 * b + 1]));
    }
    s = group_sum<kFinalThreads>(s, red);
    m = group_max<kFinalThreads>(m, redf);
    if (threadIdx.x == 0) {
        mm[0] = s / n;
        mm[1] = static_cast<double>(m);
    }
}

// Pass 2: part[2 b] = sum of (x - mean)^2, part[2 b + 1] = sum of (x - mean)^4.
__global__ __launch_bounds__(kThreads) void moments_central_kernel(
    const uint4 *__restrict__ X, int64_t chunks, const double *__restrict__ mm,
    double *__restrict__ part) {
    __shared__ double red[kThreads / 64];
    const double mean = mm[0];
    double s2 = 0.0, s4 = 0.0;
    for_chunks<true>(X, chunks, [&](const uint4 &x) {
        const float v[8] = {lo(x.x), hi(x.x), lo(x.y), hi(x.y), lo(x.z), hi(x.z), lo(x.w), hi(x.w)};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const double d = static_cast<double>(v[e]) - mean;
            const double d2 = d * d;
            s2 += d2;
            s4 += d2 * d2;
        }
    });
    s2 = group_sum<kThreads>(s2, red);
    s4 = group_sum<kThreads>(s4, red);
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = s2;
        part[2 * blockIdx.x + 1] = s4;
    }
}

// stats = [max |x|, mean, sqrt(m2), m4 / m2^2 (0 when m2 == 0)].
__global__ __launch_bounds__(kFinalThreads) void moments_final_kernel(
    const double *__restrict__ part, int blocks, double n, const double *__restrict__ mm,
    double *__restrict__ stats) {
    __shared__ double red[kFinalThreads / 64];
    double s2 = 0.0, s4 = 0.0;
    for (int b = threadIdx.x; b < blocks; b += kFinalThreads) {
        s2 += part[2 * b];
        s4 += part[2 * b + 1];
    }
    s2 = group_sum<kFinalThreads>(s2, red);
    s4 = group_sum<kFinalThreads>(s4, red);
    if (threadIdx.x == 0) {
        const double m2 = s2 / n;
        const double m4 = s4 / n;
        stats[0] = mm[1];
        stats[1] = mm[0];
        stats[2] = sqrt(m2);
        stats[3] = m2 > 0.0 ? m4 / (m2 * m2) : 0.0;
    }
}

}  // namespace

hipError_t launch_act_moments(const uint16_t *X, int64_t n, double *work, double *stats,
                              hipStream_t stream) {
    const int64_t chunks = n / 8;  // the entry point guarantees 8 | n
    const uint4 *x4 = reinterpret_cast<const uint4 *>(X);
    double *part = work;
    double *mm = work + 2 * kMomentBlocks;
    const double dn = static_cast<double>(n);
    hipLaunchKernelGGL(moments_sum_kernel, dim3(kMomentBlocks), dim3(kThreads), 0, stream, x4,
                       chunks, part);
    hipLaunchKernelGGL(moments_mean_kernel, dim3(1), dim3(kFinalThreads), 0, stream, part,
                       kMomentBlocks, dn, mm);
    hipLaunchKernelGGL(moments_central_kernel, dim3(kMomentBlocks), dim3(kThreads), 0, stream,
                       x4, chunks, mm, part);
    hipLaunchKernelGGL(moments_final_kernel, dim3(1), dim3(kFinalThreads), 0, stream, part,
                       kMomentBlocks, dn, mm, stats);
    return hipGetLastError();
}

}  // namespace w8a8
