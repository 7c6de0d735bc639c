// Fragility profile of a linear's input (paper Section 3, "Activation-
// fragility profiling and protection"): max |x|, mean, population standard
// deviation and Pearson kurtosis m4 / m2^2 over all entries of X, in binary64.
//
// One pass over X. A fixed grid of kMomentBlocks workgroups walks X in
// 16-byte chunks (8 entries) with a fixed stride; each thread takes its
// chunks kUnroll at a time (the loads first). For such a group of up to 32
// entries it computes the group's own mean and central sums of the second,
// third and fourth powers around it, from registers, and merges them into
// its running state with the pairwise update for central moments (Chan,
// Golub and LeVeque for the second; Pebay, 2008, for the third and fourth).
// Sums are never taken of raw powers, which would cancel. The threads'
// states merge in a fixed tree in LDS and each workgroup writes its state to
// the caller's workspace; one workgroup then merges the kMomentBlocks states
// in a fixed tree. Every call on the same input therefore returns the same
// bits, and X is read once, nontemporally.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "internal.h"

// Workgroup states of w8a8_act_moments_noalloc, for callers that cannot
// allocate: one file-scope device array instead of a caller workspace. Each
// GPU the library runs on holds its own copy until the process ends; host
// code never uses this name as an address (see moments_scratch below).
static __device__ __align__(256) double scratch[6 * w8a8::kMomentBlocks];

namespace w8a8 {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;      // chunk loads in flight per thread
constexpr int kStateWords = 6;  // n, mean, M2, M3, M4, max |x| (binary64 each)

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const uint4 *p) {
    const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Count, mean and central sums M_j = sum (x - mean)^j of a set of entries.
struct Moments {
    double n, mean, m2, m3, m4;
};

// 1 / n to within a few units of 2^-53: the hardware estimate refined by
// two Newton steps (fused), far shorter than a correctly rounded division.
__device__ __forceinline__ double recip(double n) {
    double r = __builtin_amdgcn_rcp(n);
    r = __builtin_fma(r, __builtin_fma(-n, r, 1.0), r);
    r = __builtin_fma(r, __builtin_fma(-n, r, 1.0), r);
    return r;
}

// The moments of the union of two disjoint sets from theirs.
__device__ __forceinline__ Moments merge(const Moments &a, const Moments &b) {
    if (b.n == 0.0) return a;
    if (a.n == 0.0) return b;
    const double n = a.n + b.n;
    const double delta = b.mean - a.mean;
    const double dn = delta * recip(n);
    const double dn2 = dn * dn;
    const double ab = a.n * b.n;
    Moments r;
    r.n = n;
    r.mean = a.mean + b.n * dn;
    r.m2 = a.m2 + b.m2 + delta * dn * ab;
    r.m3 = a.m3 + b.m3 + delta * dn2 * ab * (a.n - b.n) + 3.0 * dn * (a.n * b.m2 - b.n * a.m2);
    r.m4 = a.m4 + b.m4 + delta * dn2 * dn * ab * (a.n * a.n - ab + b.n * b.n) +
           6.0 * dn2 * (a.n * a.n * b.m2 + b.n * b.n * a.m2) + 4.0 * dn * (a.n * b.m3 - b.n * a.m3);
    return r;
}

__device__ __forceinline__ void put(double *s, int i, const Moments &m) {
    s[5 * i] = m.n;
    s[5 * i + 1] = m.mean;
    s[5 * i + 2] = m.m2;
    s[5 * i + 3] = m.m3;
    s[5 * i + 4] = m.m4;
}

__device__ __forceinline__ Moments get(const double *s, int i) {
    return Moments{s[5 * i], s[5 * i + 1], s[5 * i + 2], s[5 * i + 3], s[5 * i + 4]};
}

// Merges the NT threads' states (and maxima) of a workgroup in a fixed tree:
// at each level thread t < h takes thread t + h's state. Valid in thread 0.
// (Lane shuffles instead of LDS for the levels inside a wave measured
// slower: every lane of a wave then runs each level's merge.)
template <int NT>
__device__ __forceinline__ Moments group_merge(Moments m, float &mx, double *s, float *smx) {
    put(s, threadIdx.x, m);
    smx[threadIdx.x] = mx;
    __syncthreads();
#pragma unroll 1
    for (int h = NT / 2; h > 0; h >>= 1) {
        if (static_cast<int>(threadIdx.x) < h) {
            m = merge(m, get(s, threadIdx.x + h));
            mx = fmaxf(mx, smx[threadIdx.x + h]);
            put(s, threadIdx.x, m);
            smx[threadIdx.x] = mx;
        }
        __syncthreads();
    }
    return m;
}

// The 8 entries of a chunk, widened (exactly).
__device__ __forceinline__ void widen8(const uint4 &x, float (&v)[8]) {
    v[0] = lo(x.x);
    v[1] = hi(x.x);
    v[2] = lo(x.y);
    v[3] = hi(x.y);
    v[4] = lo(x.z);
    v[5] = hi(x.z);
    v[6] = lo(x.w);
    v[7] = hi(x.w);
}

// Pass over X: thread t of the grid takes chunks t, t + stride, ... in
// groups of kUnroll; workgroup b writes its merged state and max |x| to
// part[kStateWords b ...].
__global__ __launch_bounds__(kThreads) void moments_pass_kernel(const uint4 *__restrict__ X,
                                                                int64_t chunks,
                                                                double *__restrict__ part) {
    __shared__ double s[5 * kThreads];
    __shared__ float smx[kThreads];
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    Moments st{0.0, 0.0, 0.0, 0.0, 0.0};
    float mx = 0.0f;
    for (int64_t c0 = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; c0 < chunks;
         c0 += kUnroll * stride) {
        uint4 x[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t c = c0 + u * stride;
            x[u] = c < chunks ? load_stream(X + c) : make_uint4(0u, 0u, 0u, 0u);
        }
        int valid = 0;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) valid += c0 + u * stride < chunks ? 1 : 0;
        // the group's mean (its entries are exact in binary64; 8 valid ones
        // per chunk, and zero-filled chunks add nothing to the sum)
        double dv[kUnroll][8];
        double sum = 0.0;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            float v[8];
            widen8(x[u], v);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                dv[u][e] = static_cast<double>(v[e]);
                sum += dv[u][e];
                mx = fmaxf(mx, fabsf(v[e]));
            }
        }
        const double cnt = 8.0 * valid;
        const double gm = valid == kUnroll ? sum * (1.0 / (8.0 * kUnroll)) : sum / cnt;
        // central sums around it; the third and fourth powers accumulate
        // with fused multiply-adds (one rounding each)
        double g2 = 0.0, g3 = 0.0, g4 = 0.0;
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (u >= valid) break;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double d = dv[u][e] - gm;
                const double d2 = d * d;
                g2 += d2;
                g3 = __builtin_fma(d2, d, g3);
                g4 = __builtin_fma(d2, d2, g4);
            }
        }
        st = merge(st, Moments{cnt, gm, g2, g3, g4});
    }
    st = group_merge<kThreads>(st, mx, s, smx);
    if (threadIdx.x == 0) {
        double *o = part + kStateWords * blockIdx.x;
        o[0] = st.n;
        o[1] = st.mean;
        o[2] = st.m2;
        o[3] = st.m3;
        o[4] = st.m4;
        o[5] = static_cast<double>(mx);
    }
}

// stats = [max |x|, mean, sqrt(m2), m4 / m2^2 (0 when m2 == 0)] from the
// kMomentBlocks workgroup states, merged in a fixed tree.
__global__ __launch_bounds__(kMomentBlocks) void moments_final_kernel(
    const double *__restrict__ part, double *__restrict__ stats) {
    __shared__ double s[5 * kMomentBlocks];
    __shared__ float smx[kMomentBlocks];
    const double *p = part + kStateWords * threadIdx.x;
    Moments m{p[0], p[1], p[2], p[3], p[4]};
    float mx = static_cast<float>(p[5]);
    m = group_merge<kMomentBlocks>(m, mx, s, smx);
    if (threadIdx.x == 0) {
        const double m2 = m.m2 / m.n;
        const double m4 = m.m4 / m.n;
        stats[0] = static_cast<double>(mx);
        stats[1] = m.mean;
        stats[2] = sqrt(m2);
        stats[3] = m2 > 0.0 ? m4 / (m2 * m2) : 0.0;
    }
}

}  // namespace

namespace {

// Device address of `scratch` on each GPU, looked up once per device with
// that device current (each GPU has its own copy at its own address).
constexpr int kMaxDevices = 256;
std::atomic<double *> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

hipError_t moments_scratch(double **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    double *p = g_scratch[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            void *q = nullptr;
            e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (q == nullptr) return hipErrorInvalidSymbol;
            p = static_cast<double *>(q);
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return hipSuccess;
}

}  // namespace

static_assert(sizeof(scratch) == 6 * kMomentBlocks * sizeof(double), "scratch size");

hipError_t launch_act_moments_noalloc(const uint16_t *X, int64_t n, double *stats,
                                      hipStream_t stream) {
    double *work = nullptr;
    const hipError_t e = moments_scratch(&work);
    if (e != hipSuccess) return e;
    // Every workgroup of the pass writes its state before the final merge
    // reads it (stream order), so nothing needs clearing between calls.
    return launch_act_moments(X, n, work, stats, stream);
}

hipError_t launch_act_moments(const uint16_t *X, int64_t n, double *work, double *stats,
                              hipStream_t stream) {
    const int64_t chunks = n / 8;  // the entry point guarantees 8 | n
    hipLaunchKernelGGL(moments_pass_kernel, dim3(kMomentBlocks), dim3(kThreads), 0, stream,
                       reinterpret_cast<const uint4 *>(X), chunks, work);
    hipLaunchKernelGGL(moments_final_kernel, dim3(1), dim3(kMomentBlocks), 0, stream, work,
                       stats);
    return hipGetLastError();
}

}  // namespace w8a8
