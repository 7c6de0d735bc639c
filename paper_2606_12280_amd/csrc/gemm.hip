// MFMA GEMMs of the W8A8 linear for gfx950 (CDNA4), paper Section 3:
//   - INT8 x INT8 -> INT32 with the dequantization + bias epilogue fused in
//     registers (the fused INT8 GEMM the paper's Section 7 names as missing);
//   - bf16 x bf16 -> fp32 for the protected layers.
//
// Both operands are K-contiguous ("NT": X [M][K], W [N][K]), the natural
// layout for MFMA, where each lane feeds 16 contiguous bytes of one row per
// instruction. The skeleton works on 16-byte chunks along K, so one kernel
// serves both element types: v_mfma_i32_32x32x32_i8 consumes 32 int8 per row
// and v_mfma_f32_32x32x16_bf16 16 bf16 per row, i.e. two chunks either way.
//
// Structure of one workgroup (BM x BN output tile, WAVES_M x WAVES_N waves):
//   global -> registers: range-checked buffer loads (rows past M/N and the K
//     tail read as zero, so ragged tiles need no branches);
//   registers -> LDS: double-buffered tiles with an XOR swizzle of the
//     16-byte chunks so that the fragment reads are free of bank conflicts;
//   LDS -> registers -> MFMA: each wave owns a WM x WN sub-tile made of
//     32x32 MFMA blocks, accumulators in (A)VGPRs;
//   epilogue: float(acc) * (x_scale[m] * w_scale[n]) + bias[n] -> bf16 with
//     a range-checked buffer store.
// The next K tile is loaded into registers while the current one is being
// multiplied; one barrier per K tile.
//
// Launch order is XCD-aware: workgroups are dispatched round-robin over the
// 8 XCDs, so block id b runs on XCD b % 8. Each XCD is given a contiguous
// range of tiles, walked in groups of GROUP_M tile rows, so that the tiles
// resident on one XCD at a time share A and B panels in that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace w8a8 {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format
constexpr uint32_t kOutOfRange = 0x80000000u;  // any offset past num_records

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, static_cast<int>(bytes),
                                             kBufferWord3);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));  // v_cvt_pk_bf16_f32 (RNE)
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

struct I8Op {
    using Acc = v16i;
    __device__ static Acc mma(v4i a, v4i b, Acc c) {
        return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
    }
};

struct Bf16Op {
    using Acc = v16f;
    __device__ static Acc mma(v4i a, v4i b, Acc c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a),
                                                       __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
    }
};

enum Epilogue { kDequantBf16 = 0, kStoreI32 = 1, kBiasBf16 = 2 };

template <int GROUP_M>
__device__ __forceinline__ void map_tile(int pid, int tiles_m, int tiles_n, int &tm, int &tn) {
    constexpr int kXcd = 8;
    const int total = tiles_m * tiles_n;
    const int full = total - total % kXcd;
    int lid = pid;
    if (pid < full) lid = (pid % kXcd) * (full / kXcd) + pid / kXcd;
    const int group = GROUP_M * tiles_n;
    const int g = lid / group;
    const int first_m = g * GROUP_M;
    const int gm = min(tiles_m - first_m, GROUP_M);
    const int in = lid - g * group;
    tm = first_m + in % gm;
    tn = in / gm;
}

template <class Op, int BM, int BN, int BKB, int WAVES_M, int WAVES_N, int SWZ_SHIFT,
          int GROUP_M, int EPI>
__global__ __launch_bounds__(WAVES_M *WAVES_N * 64) void gemm_kernel(
    const int8_t *__restrict__ A, const int8_t *__restrict__ B, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int NT = WAVES_M * WAVES_N * 64;
    constexpr int WM = BM / WAVES_M;
    constexpr int WN = BN / WAVES_N;
    constexpr int TM = WM / 32;
    constexpr int TN = WN / 32;
    constexpr int CPR = BKB / 16;        // 16-byte chunks per tile row
    constexpr int RSTEP = NT / CPR;      // tile rows covered by one load round
    constexpr int A_LOADS = BM / RSTEP;
    constexpr int B_LOADS = BN / RSTEP;
    constexpr int KSTEPS = BKB / 32;     // MFMA steps per K tile (2 chunks each)
    constexpr int STAGE = (BM + BN) * BKB;
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(NT % CPR == 0 && BM % RSTEP == 0 && BN % RSTEP == 0, "load split");
    static_assert(RSTEP % 32 == 0, "swizzle key must not depend on the load round");
    static_assert(CPR == 4 || CPR == 8, "K tile of 64 or 128 bytes");

    __shared__ __attribute__((aligned(16))) int8_t smem[2 * STAGE];

    int tm, tn;
    map_tile<GROUP_M>(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;

    // Range-checked views of this tile's row panels: rows past M (N) and
    // offsets marked out of range load as zero.
    const int rows_a = min(BM, M - m0);
    const int rows_b = min(BN, N - n0);
    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(A + static_cast<int64_t>(m0) * Kb, static_cast<uint32_t>(rows_a) * Kb);
    const __amdgpu_buffer_rsrc_t rb =
        make_rsrc(B + static_cast<int64_t>(n0) * Kb, static_cast<uint32_t>(rows_b) * Kb);

    // This thread's chunk column and first row inside the tile.
    const int lc = tid % CPR;
    const int lr = tid / CPR;
    const int lswz = lc ^ ((lr >> SWZ_SHIFT) & (CPR - 1));
    const uint32_t g_off = static_cast<uint32_t>(lr) * Kb + lc * 16;
    const int lds_off = lr * BKB + lswz * 16;

    v4i sa[A_LOADS];
    v4i sb[B_LOADS];
    const int KT = (Kb + BKB - 1) / BKB;

    auto gload = [&](int kt) {
        const int kb = kt * BKB;
        const bool ok = kb + lc * 16 < Kb;  // K tail (Kb % 64 == 0)
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
            const uint32_t off = ok ? g_off + static_cast<uint32_t>(i * RSTEP) * Kb + kb : kOutOfRange;
            sa[i] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, 0));
        }
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i) {
            const uint32_t off = ok ? g_off + static_cast<uint32_t>(i * RSTEP) * Kb + kb : kOutOfRange;
            sb[i] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rb, off, 0, 0));
        }
    };
    auto lstore = [&](int stage) {
        int8_t *base = smem + stage * STAGE;
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i)
            *reinterpret_cast<v4i *>(base + lds_off + i * RSTEP * BKB) = sa[i];
#pragma unroll
        for (int i = 0; i < B_LOADS; ++i)
            *reinterpret_cast<v4i *>(base + BM * BKB + lds_off + i * RSTEP * BKB) = sb[i];
    };

    // Fragment addressing: lane reads row (lane % 32) of each 32-row block,
    // chunk 2*s + lane/32 of the K tile.
    const int frow = lane & 31;
    const int fhalf = lane >> 5;
    const int fkey = (frow >> SWZ_SHIFT) & (CPR - 1);  // same for every 32-row block
    const int a_row_base = (wm * WM + frow) * BKB;
    const int b_row_base = BM * BKB + (wn * WN + frow) * BKB;

    typename Op::Acc acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = typename Op::Acc{};

    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT) gload(kt + 1);
        const int8_t *base = smem + cur * STAGE;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
            const int chunk = (2 * s + fhalf) ^ fkey;
            v4i af[TM];
            v4i bf[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                af[i] = *reinterpret_cast<const v4i *>(base + a_row_base + i * 32 * BKB + chunk * 16);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                bf[j] = *reinterpret_cast<const v4i *>(base + b_row_base + j * 32 * BKB + chunk * 16);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) acc[i][j] = Op::mma(af[i], bf[j], acc[i][j]);
        }
        if (kt + 1 < KT) lstore(cur ^ 1);
        __syncthreads();
    }

    // Epilogue. Accumulator element r of block (i, j) in lane l holds
    // row 32i + 8(r/4) + 4(l/32) + r%4 and column 32j + l%32 of the wave tile.
    const int ncol0 = n0 + wn * WN + frow;
    const int mrow0 = m0 + wm * WM + 4 * fhalf;
    const uint32_t ybytes = EPI == kStoreI32 ? 4u : 2u;
    const __amdgpu_buffer_rsrc_t ry =
        make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * ybytes,
                  static_cast<uint32_t>(rows_a) * N * ybytes);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        float xrow[16];
        if constexpr (EPI == kDequantBf16) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = mrow0 + 32 * i + 8 * (r >> 2) + (r & 3);
                xrow[r] = m < M ? xs[m] : 0.0f;
            }
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = ncol0 + 32 * j;
            const bool n_ok = n < N;
            float wsn = 0.0f;
            float bn = 0.0f;
            if constexpr (EPI == kDequantBf16) {
                if (n_ok) wsn = ws[n];
            }
            if constexpr (EPI != kStoreI32) {
                if (n_ok && bias != nullptr) bn = bf16_bits_to_f32(bias[n]);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int ml = mrow0 - m0 + 32 * i + 8 * (r >> 2) + (r & 3);  // row in tile
                const uint32_t off =
                    n_ok ? (static_cast<uint32_t>(ml) * N + n) * ybytes : kOutOfRange;
                if constexpr (EPI == kStoreI32) {
                    __builtin_amdgcn_raw_buffer_store_b32(acc[i][j][r], ry, off, 0, 0);
                } else if constexpr (EPI == kDequantBf16) {
                    const float y = __builtin_fmaf(static_cast<float>(acc[i][j][r]),
                                                   xrow[r] * wsn, bn);
                    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(y), ry, off, 0, 0);
                } else {
                    const float y = acc[i][j][r] + bn;
                    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(y), ry, off, 0, 0);
                }
            }
        }
    }
}

template <class Op, int BM, int BN, int BKB, int WAVES_M, int WAVES_N, int SWZ_SHIFT,
          int GROUP_M, int EPI>
hipError_t launch(const int8_t *A, const int8_t *B, const float *xs, const float *ws,
                  const uint16_t *bias, int64_t M, int64_t N, int64_t Kb, void *Y,
                  hipStream_t stream) {
    const int tiles_m = static_cast<int>((M + BM - 1) / BM);
    const int tiles_n = static_cast<int>((N + BN - 1) / BN);
    const int64_t blocks = static_cast<int64_t>(tiles_m) * tiles_n;
    hipLaunchKernelGGL(
        (gemm_kernel<Op, BM, BN, BKB, WAVES_M, WAVES_N, SWZ_SHIFT, GROUP_M, EPI>),
        dim3(static_cast<unsigned>(blocks)), dim3(WAVES_M * WAVES_N * 64), 0, stream, A, B, xs,
        ws, bias, static_cast<int>(M), static_cast<int>(N), static_cast<int>(Kb), Y, tiles_m,
        tiles_n);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_i8(const int8_t *A, const int8_t *B, const float *xs, const float *ws,
                          const uint16_t *bias, int64_t M, int64_t N, int64_t K, uint16_t *Y,
                          int32_t *Y32, hipStream_t stream) {
    if (Y32 != nullptr)
        return launch<I8Op, 256, 128, 128, 2, 2, 0, 4, kStoreI32>(A, B, nullptr, nullptr, nullptr,
                                                                  M, N, K, Y32, stream);
    return launch<I8Op, 256, 128, 128, 2, 2, 0, 4, kDequantBf16>(A, B, xs, ws, bias, M, N, K, Y,
                                                                 stream);
}

hipError_t launch_gemm_bf16(const uint16_t *A, const uint16_t *B, const uint16_t *bias,
                            int64_t M, int64_t N, int64_t K, uint16_t *Y, hipStream_t stream) {
    return launch<Bf16Op, 256, 128, 128, 2, 2, 0, 4, kBiasBf16>(
        reinterpret_cast<const int8_t *>(A), reinterpret_cast<const int8_t *>(B), nullptr, nullptr,
        bias, M, N, 2 * K, Y, stream);
}

}  // namespace w8a8
