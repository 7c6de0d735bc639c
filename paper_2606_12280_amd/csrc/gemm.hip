// MFMA GEMMs of the W8A8 linear for gfx950 (CDNA4), paper Section 3:
//   - INT8 x INT8 -> INT32 with the dequantization + bias epilogue fused in
//     registers (the fused INT8 GEMM the paper's Section 7 names as missing);
//   - bf16 x bf16 -> fp32 for the protected layers.
//
// Both operands are K-contiguous ("NT": X [M][K], W [N][K]), the natural
// layout for MFMA, where each lane feeds 16 contiguous bytes of one row per
// instruction. The kernel works on 16-byte chunks along K, so one skeleton
// serves both element types: v_mfma_i32_32x32x32_i8 consumes 32 int8 of a row
// and v_mfma_f32_32x32x16_bf16 16 bf16, i.e. two chunks either way.
//
// One workgroup computes a BM x BN tile of Y with WAVES_M x WAVES_N waves.
//
//   global -> LDS: direct-to-LDS buffer loads (buffer_load_dwordx4 ... lds),
//     no VGPR staging. Each wave instruction fills 1 KiB of LDS; the global
//     address of every lane is chosen so that the 16-byte chunks land
//     XOR-swizzled (chunk c of row r at chunk c ^ ((r >> SWZ) & (CPR-1))),
//     which keeps the fragment reads free of bank conflicts. The loads are
//     range-checked: rows past M/N and the K tail read as zero.
//   pipeline: a ring of STAGES K-tiles in LDS; STAGES-1 tiles are in flight
//     while one is multiplied. Waits are explicit (s_waitcnt vmcnt(n) on the
//     wave's own loads, then s_barrier for the other waves'), so prefetches
//     stay in flight across iterations. MFMA fragments are double-buffered
//     in registers: the next step's LDS reads overlap the current MFMAs, also
//     across the tile boundary.
//   MFMA: the W tile feeds the instruction's first operand and the X tile
//     its second, so C = W X^T and lane l holds token m = l % 32 of a 32x32
//     block with 4 consecutive output channels per accumulator quad.
//   epilogue: y = float(acc) * (x_scale[m] * w_scale[n]) + bias[n] with one
//     fma, four channels packed into 8 bytes of bf16 per store.
//
// Launch order is XCD-aware: workgroups are dispatched round-robin over the
// 8 XCDs, so block id b runs on XCD b % 8. Each XCD is given a contiguous
// range of tiles, walked GROUP_M tile rows at a time, so that the tiles
// resident on one XCD share X and W panels in that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "internal.h"

namespace w8a8 {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

#define LDS_AS __attribute__((address_space(3)))

constexpr int kBufferWord3 = 0x00020000;       // raw buffer, 32-bit data format
constexpr uint32_t kOutOfRange = 0x80000000u;  // past any num_records used here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, static_cast<int>(bytes),
                                             kBufferWord3);
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));  // v_cvt_pk_bf16_f32 (RNE)
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt[3:0] in bits
// 3:0 and vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

// Workgroup barrier without a memory fence: a fence would drain every
// outstanding global load, i.e. the prefetch pipeline. Ordering of LDS
// accesses around it is by the explicit waits; the empty asm statements keep
// the compiler from moving memory operations across.
__device__ __forceinline__ void barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
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

template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int SWZ,
          int GROUP_M, int EPI, bool N_VEC, bool HAS_BIAS>
__global__ __launch_bounds__(WAVES_M *WAVES_N * 64) void gemm_kernel(
    const int8_t *__restrict__ X, const int8_t *__restrict__ W, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int WTM = BM / WAVES_M;   // tokens per wave
    constexpr int WTN = BN / WAVES_N;   // channels per wave
    constexpr int TJ = WTM / 32;        // 32-token blocks per wave
    constexpr int TI = WTN / 32;        // 32-channel blocks per wave
    constexpr int CPR = BK / 16;        // 16-byte chunks per tile row
    constexpr int ROWS_PER_KB = 1024 / BK;
    constexpr int LA = BM * BK / 1024 / NW;  // 1 KiB DMA blocks per wave, X tile
    constexpr int LB = BN * BK / 1024 / NW;  // ... W tile
    constexpr int LOADS = LA + LB;
    constexpr int KSTEPS = BK / 32;
    constexpr int STAGE = (BM + BN) * BK;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(LA * NW * 1024 == BM * BK && LB * NW * 1024 == BN * BK, "DMA split");
    static_assert(CPR == 4 || CPR == 8, "K tile of 64 or 128 bytes");
    static_assert(STAGES >= 2 && LOADS * (STAGES - 2) < 64, "vmcnt range");
    static_assert(KSTEPS % 2 == 0, "fragment buffer 0 starts every tile");
    static_assert(STAGES * STAGE <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) int8_t smem[STAGES * STAGE];

    // Materialize the epilogue's pointer arguments now: a scalar load of a
    // kernel argument left pending into the main loop would make every LDS
    // wait there a full lgkmcnt(0) (scalar loads complete out of order).
    asm volatile("" ::"s"(xs), "s"(ws), "s"(bias), "s"(Yout));

    int tm, tn;
    map_tile<GROUP_M>(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;

    const int rows_x = min(BM, M - m0);
    const int rows_w = min(BN, N - n0);

    // Epilogue operands of this lane, loaded up front (before the tile loads,
    // so that the in-order vmcnt accounting below is unaffected): x_scale of
    // its TJ tokens, w_scale and bias of its TI x 4 x 4 channels. Channel
    // quad g of block i is n = n0 + wn*WTN + 32 i + 8 g + 4 (l / 32) + e.
    const int frow = lane & 31;
    const int fhalf = lane >> 5;
    float ep_xs[TJ];
    float ep_ws[TI][4][4];
    uint32_t ep_b[TI][4][2];  // bf16 pairs, converted in the epilogue
    {
        // Range-checked loads (zero past M / N, or for a missing bias): no
        // branch, and nothing consumes them before the epilogue, so the
        // compiler waits for them only there.
        const __amdgpu_buffer_rsrc_t rxs =
            make_rsrc(EPI == kDequantBf16 ? xs + m0 : nullptr,
                      EPI == kDequantBf16 ? static_cast<uint32_t>(rows_x) * 4u : 0u);
        const __amdgpu_buffer_rsrc_t rws =
            make_rsrc(ws, EPI == kDequantBf16 ? static_cast<uint32_t>(N) * 4u : 0u);
        const __amdgpu_buffer_rsrc_t rbs =
            make_rsrc(bias, HAS_BIAS ? static_cast<uint32_t>(N) * 2u : 0u);
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            const uint32_t ml = wm * WTM + 32 * j + frow;
            ep_xs[j] = __builtin_bit_cast(float,
                                          __builtin_amdgcn_raw_buffer_load_b32(rxs, ml * 4u, 0, 0));
        }
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t n = n0 + wn * WTN + 32 * i + 8 * g + 4 * fhalf;
                if constexpr (N_VEC) {
                    // N % 4 == 0 (and w_scale / bias aligned): the 4 channels are all
                    // inside or all outside; outside, a valid address is read and
                    // discarded. (Plain vector loads: extracting the elements of a
                    // 128-bit buffer load through bit casts miscompiles with this
                    // compiler, which narrows the load to its first dword.)
                    const bool ok = static_cast<int>(n) < N;
                    const uint32_t nc = ok ? n : 0u;
                    if constexpr (EPI == kDequantBf16) {
                        const float4 w4 = *reinterpret_cast<const float4 *>(ws + nc);
                        ep_ws[i][g][0] = ok ? w4.x : 0.0f;
                        ep_ws[i][g][1] = ok ? w4.y : 0.0f;
                        ep_ws[i][g][2] = ok ? w4.z : 0.0f;
                        ep_ws[i][g][3] = ok ? w4.w : 0.0f;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) ep_ws[i][g][e] = 0.0f;
                    }
                    ep_b[i][g][0] = 0u;
                    ep_b[i][g][1] = 0u;
                    if constexpr (HAS_BIAS) {
                        const uint2 b2 = *reinterpret_cast<const uint2 *>(bias + nc);
                        ep_b[i][g][0] = ok ? b2.x : 0u;
                        ep_b[i][g][1] = ok ? b2.y : 0u;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        ep_ws[i][g][e] = __builtin_bit_cast(
                            float, __builtin_amdgcn_raw_buffer_load_b32(rws, (n + e) * 4u, 0, 0));
#pragma unroll
                    for (int h = 0; h < 2; ++h)
                        ep_b[i][g][h] =
                            __builtin_amdgcn_raw_buffer_load_b16(rbs, (n + 2 * h) * 2u, 0, 0) |
                            static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(
                                rbs, (n + 2 * h + 1) * 2u, 0, 0))
                                << 16;
                }
            }
    }
    // These loads must stay older than every tile load: the vmcnt waits of
    // the pipeline below count only tile loads as younger. (They are global
    // loads and the tile loads write LDS, so nothing else orders them.)
    __builtin_amdgcn_sched_barrier(0);

    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(X + static_cast<int64_t>(m0) * Kb, static_cast<uint32_t>(rows_x) * Kb);
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(W + static_cast<int64_t>(n0) * Kb, static_cast<uint32_t>(rows_w) * Kb);

    // DMA source offsets. Lane l of the wave's i-th block writes LDS bytes
    // [blk*1024 + 16 l, +16) = row (blk*ROWS_PER_KB + l / CPR), physical
    // chunk l % CPR, which holds logical chunk (l % CPR) ^ swizzle(row).
    const int dma_row = lane / CPR;
    const int dma_phys = lane % CPR;
    uint32_t off_x[LA], off_w[LB];
    int chunk_x[LA], chunk_w[LB];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int row = (wave + i * NW) * ROWS_PER_KB + dma_row;
        chunk_x[i] = dma_phys ^ ((row >> SWZ) & (CPR - 1));
        off_x[i] = static_cast<uint32_t>(row) * Kb + chunk_x[i] * 16;
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int row = (wave + i * NW) * ROWS_PER_KB + dma_row;
        chunk_w[i] = dma_phys ^ ((row >> SWZ) & (CPR - 1));
        off_w[i] = static_cast<uint32_t>(row) * Kb + chunk_w[i] * 16;
    }

    const int KT = (Kb + BK - 1) / BK;
    auto issue = [&](int kt) {
        int8_t *slot = smem + (kt % STAGES) * STAGE;
        const int kb = kt * BK;
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const uint32_t off = kb + chunk_x[i] * 16 < Kb ? off_x[i] + kb : kOutOfRange;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rx, (LDS_AS void *)(slot + (wave + i * NW) * 1024), 16, off, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const uint32_t off = kb + chunk_w[i] * 16 < Kb ? off_w[i] + kb : kOutOfRange;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rw, (LDS_AS void *)(slot + BM * BK + (wave + i * NW) * 1024), 16, off, 0, 0, 0);
        }
    };

    // Fragment reads: lane reads row (l % 32) of a 32-row block, chunk
    // 2 s + l / 32 of the K tile; the swizzle key depends on l only.
    const int fkey = (frow >> SWZ) & (CPR - 1);
    const int x_base = (wm * WTM + frow) * BK;
    const int w_base = BM * BK + (wn * WTN + frow) * BK;

    typename Op::Acc acc[TI][TJ];
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = typename Op::Acc{};

    // Fragments of one MFMA step, double-buffered: the next step's are read
    // from LDS while the current step's MFMAs run.
    v4i wf[2][TI];
    v4i xf[2][TJ];
    auto load_frags = [&](const int8_t *slot, int s, v4i(&wb)[TI], v4i(&xb)[TJ]) {
        const int chunk = (2 * s + fhalf) ^ fkey;
#pragma unroll
        for (int i = 0; i < TI; ++i)
            wb[i] = *reinterpret_cast<const v4i *>(slot + w_base + i * 32 * BK + chunk * 16);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
            xb[j] = *reinterpret_cast<const v4i *>(slot + x_base + j * 32 * BK + chunk * 16);
    };

    auto mfma_step = [&](int cur) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int j = 0; j < TJ; ++j) acc[i][j] = Op::mma(wf[cur][i], xf[cur][j], acc[i][j]);
    };

    // One K tile. Steps 0..KSTEPS-2 read the next step's fragments, then run
    // the current MFMAs. Before the last step comes the tile boundary: every
    // read of tile kt has completed (the last ones were issued a whole MFMA
    // step ago); once this wave's loads of tile kt+1 are in and all waves
    // meet, slot kt is refilled with tile kt+STAGES (ISSUE) and tile kt+1's
    // first fragments are read. Scheduling barriers keep each group of reads
    // ahead of the MFMAs it overlaps (the compiler would otherwise sink the
    // reads to their uses), and the loops below are branch-free so that the
    // compiler's own waits stay exact (lgkmcnt(n) on the older reads only).
    auto tile = [&](int kt, auto issue_tag, auto vm_tag, auto last_tag) {
        constexpr bool ISSUE = decltype(issue_tag)::value;
        constexpr int VM = decltype(vm_tag)::value;
        constexpr bool LAST = decltype(last_tag)::value;
        const int8_t *slot = smem + (kt % STAGES) * STAGE;
#pragma unroll
        for (int s = 0; s + 1 < KSTEPS; ++s) {
            load_frags(slot, s + 1, wf[(s + 1) & 1], xf[(s + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            mfma_step(s & 1);
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (!LAST) {
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
            wait_vmcnt<VM>();
            barrier();
            if constexpr (ISSUE) issue(kt + STAGES);
            load_frags(smem + ((kt + 1) % STAGES) * STAGE, 0, wf[0], xf[0]);
            __builtin_amdgcn_sched_barrier(0);
        }
        mfma_step((KSTEPS - 1) & 1);
        __builtin_amdgcn_sched_barrier(0);
    };
    using T = std::true_type;
    using F = std::false_type;
    using VM_STEADY = std::integral_constant<int, LOADS * (STAGES - 2)>;
    using VM_ALL = std::integral_constant<int, 0>;

    // Prologue: tiles 0..STAGES-2 in flight; once tile 0 has landed the last
    // slot is issued too and the first fragments are read.
#pragma unroll
    for (int t = 0; t < STAGES - 1; ++t)
        if (t < KT) issue(t);
    if (STAGES - 1 <= KT)
        wait_vmcnt<LOADS * (STAGES - 2)>();
    else
        wait_vmcnt<0>();
    barrier();
    if (STAGES - 1 < KT) issue(STAGES - 1);
    load_frags(smem, 0, wf[0], xf[0]);

    int kt = 0;
    for (; kt + STAGES < KT; ++kt) tile(kt, T{}, VM_STEADY{}, F{});   // refill as we go
    for (; kt + 1 < KT; ++kt) tile(kt, F{}, VM_ALL{}, F{});           // drain the ring
    tile(kt, F{}, VM_ALL{}, T{});                                     // last tile

    // Epilogue. In block (i, j), accumulator element r of lane l holds
    // channel 32 i + 8 (r / 4) + 4 (l / 32) + r % 4 and token 32 j + l % 32
    // of the wave tile: each quad r = 4g..4g+3 is 4 consecutive channels.
    constexpr uint32_t kYBytes = EPI == kStoreI32 ? 4u : 2u;
    const __amdgpu_buffer_rsrc_t ry =
        make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * kYBytes,
                  static_cast<uint32_t>(rows_x) * N * kYBytes);
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
        const int ml = wm * WTM + 32 * j + frow;  // token within the tile
        const uint32_t row_off = static_cast<uint32_t>(ml) * N;
#pragma unroll
        for (int i = 0; i < TI; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = n0 + wn * WTN + 32 * i + 8 * g + 4 * fhalf;
                if constexpr (EPI == kStoreI32) {
                    if (N_VEC && n + 3 < N) {
                        const v4i v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                       acc[i][j][4 * g + 3]};
                        __builtin_amdgcn_raw_buffer_store_b128(v, ry, (row_off + n) * 4u, 0, 0);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t off = n + e < N ? (row_off + n + e) * 4u : kOutOfRange;
                            __builtin_amdgcn_raw_buffer_store_b32(acc[i][j][4 * g + e], ry, off, 0,
                                                                  0);
                        }
                    }
                } else {
                    uint32_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float a = static_cast<float>(acc[i][j][4 * g + e]);
                        float y;
                        const uint32_t bw = ep_b[i][g][e >> 1];
                        const float b = __uint_as_float((e & 1) ? (bw & 0xffff0000u) : (bw << 16));
                        if constexpr (EPI == kDequantBf16)
                            y = __builtin_fmaf(a, ep_xs[j] * ep_ws[i][g][e], b);
                        else
                            y = a + b;
                        h[e] = f32_to_bf16_bits(y);
                    }
                    if (N_VEC && n + 3 < N) {
                        const v2u v = {h[0] | h[1] << 16, h[2] | h[3] << 16};
                        __builtin_amdgcn_raw_buffer_store_b64(v, ry, (row_off + n) * 2u, 0, 0);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t off = n + e < N ? (row_off + n + e) * 2u : kOutOfRange;
                            __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h[e]), ry,
                                                                  off, 0, 0);
                        }
                    }
                }
            }
        }
    }
}

template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int SWZ,
          int GROUP_M, int EPI>
hipError_t launch(const int8_t *X, const int8_t *W, const float *xs, const float *ws,
                  const uint16_t *bias, int64_t M, int64_t N, int64_t Kb, void *Y,
                  hipStream_t stream) {
    const int tiles_m = static_cast<int>((M + BM - 1) / BM);
    const int tiles_n = static_cast<int>((N + BN - 1) / BN);
    const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(tiles_m) * tiles_n));
    const dim3 block(WAVES_M * WAVES_N * 64);
    const bool has_bias = EPI != kStoreI32 && bias != nullptr;
    const bool n_vec = N % 4 == 0 && (reinterpret_cast<uintptr_t>(ws) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(bias) & 7) == 0;
    const int iM = static_cast<int>(M), iN = static_cast<int>(N), iK = static_cast<int>(Kb);
#define W8A8_LAUNCH(NV, HB)                                                                     \
    hipLaunchKernelGGL(                                                                          \
        (gemm_kernel<Op, BM, BN, BK, WAVES_M, WAVES_N, STAGES, SWZ, GROUP_M, EPI, NV, HB>), grid, \
        block, 0, stream, X, W, xs, ws, bias, iM, iN, iK, Y, tiles_m, tiles_n)
    if (n_vec && has_bias)
        W8A8_LAUNCH(true, true);
    else if (n_vec)
        W8A8_LAUNCH(true, false);
    else if (has_bias)
        W8A8_LAUNCH(false, true);
    else
        W8A8_LAUNCH(false, false);
#undef W8A8_LAUNCH
    return hipGetLastError();
}

// 192 x 256 tiles (tokens x channels), four waves of 192 x 64, 4-stage ring of
// 64-byte K tiles, chunk swizzle key (row >> 2) & 3 (conflict-free for the
// 64-bank LDS, which serves a 16-byte read for 16 lanes per cycle), groups of
// 4 tile rows. At M = 4608 the DiT FFN up-projection is 24 x 64 tiles: six
// full rounds of the 256 CUs.
#define W8A8_GEMM_CFG 192, 256, 64, 1, 4, 4, 2, 4

}  // namespace

hipError_t launch_gemm_i8(const int8_t *A, const int8_t *B, const float *xs, const float *ws,
                          const uint16_t *bias, int64_t M, int64_t N, int64_t K, uint16_t *Y,
                          int32_t *Y32, hipStream_t stream) {
    if (Y32 != nullptr)
        return launch<I8Op, W8A8_GEMM_CFG, kStoreI32>(A, B, nullptr, nullptr, nullptr, M, N, K,
                                                      Y32, stream);
    return launch<I8Op, W8A8_GEMM_CFG, kDequantBf16>(A, B, xs, ws, bias, M, N, K, Y, stream);
}

hipError_t launch_gemm_bf16(const uint16_t *A, const uint16_t *B, const uint16_t *bias,
                            int64_t M, int64_t N, int64_t K, uint16_t *Y, hipStream_t stream) {
    return launch<Bf16Op, W8A8_GEMM_CFG, kBiasBf16>(
        reinterpret_cast<const int8_t *>(A), reinterpret_cast<const int8_t *>(B), nullptr, nullptr,
        bias, M, N, 2 * K, Y, stream);
}

}  // namespace w8a8
