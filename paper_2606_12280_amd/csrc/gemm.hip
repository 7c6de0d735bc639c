// MFMA GEMMs of the W8A8 linear for gfx950 (CDNA4), paper Section 3:
//   - INT8 x INT8 -> INT32 with the dequantization + bias epilogue fused in
//     registers (the fused INT8 GEMM the paper's Section 7 names as missing);
//   - bf16 x bf16 -> fp32 for the protected layers.
//
// Both operands are K-contiguous ("NT": X [M][K], W [N][K]), the natural
// layout for MFMA, where each lane feeds 16 contiguous bytes of one row per
// instruction. The kernels work on 16-byte chunks along K, so one skeleton
// serves both element types. The 12-wave kernels multiply 16 x 16 blocks
// with a 64-byte K step (v_mfma_i32_16x16x64_i8: 64 int8 of a row,
// v_mfma_f32_16x16x32_bf16: 32 bf16, four chunks either way); the others
// 32 x 32 blocks with a 32-byte step (v_mfma_i32_32x32x32_i8,
// v_mfma_f32_32x32x16_bf16, two chunks). Under the GPU's power limit the
// 16 x 16 forms hold a higher clock: they move half the accumulator bytes
// per multiply-add.
//
// A workgroup computes a BM x BN tile of Y.
//
//   global -> LDS: direct-to-LDS buffer loads (buffer_load_dwordx4 ... lds),
//     no VGPR staging. Each wave instruction fills 1 KiB of LDS; the global
//     address of every lane is chosen so that the 16-byte chunks land
//     XOR-swizzled (chunk c of row r at chunk c ^ ((r >> SWZ) & (CPR-1))).
//     The LDS has 64 banks and serves a 16-byte read for 16 lanes per cycle,
//     i.e. 256 bytes = 256/BK rows, so SWZ = log2(256/BK) makes the fragment
//     reads conflict-free. Loads are range-checked: rows past M/N read as 0.
//   pipeline: a ring of STAGES K tiles in LDS. Waits are explicit
//     (s_waitcnt vmcnt(n) on a wave's own loads, then s_barrier without a
//     memory fence, which would drain every prefetch).
//   MFMA: the W tile feeds the instruction's first operand and the X tile
//     its second, so C = W X^T; every accumulator quad holds 4 consecutive
//     output channels of one token (lane l: token l % 32 of a 32 x 32 block,
//     or l % 16 of a 16 x 16 block). Fragments are read ahead into
//     registers: the next step's LDS reads overlap the current MFMAs, also
//     across tile boundaries.
//   epilogue: y = float(acc) * (x_scale[m] * w_scale[n]) + bias[n] with one
//     fma, four channels packed into 8 bytes of bf16 per store.
//
// Three kernels share this skeleton:
//   gemm_2s_kernel  large tiles (288 x 256 with 12 waves, 192 x 256 with 8)
//                   in two-slot rings; four of the waves also issue the tile
//                   loads. The default wherever its tiles fill the CUs, and
//                   made persistent as gemm_pt_kernel where they take more
//                   than one round of the CUs;
//   gemm_ws_kernel  warp-specialized: NPROD producer waves only issue the
//                   tile loads, the WAVES_M x WAVES_N consumer waves only read
//                   fragments and run MFMAs. With one wave doing both, the
//                   in-order issue stalls the MFMA stream whenever the load
//                   path pushes back; split across waves that share a SIMD,
//                   loads and MFMAs proceed side by side. Small outputs;
//   gemm_kernel     every wave loads and multiplies (used when the K tile is
//                   64 bytes, i.e. K not a multiple of 128 bytes).
//
// Launch order is XCD-aware: workgroups are dispatched round-robin over the
// 8 XCDs, so block id b runs on XCD b % 8. Each XCD is given a contiguous
// range of tiles, walked GROUP_M tile rows at a time, so that the tiles
// resident on one XCD share X and W panels in that XCD's L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

#include "internal.h"

namespace w8a8 {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

#define LDS_AS __attribute__((address_space(3)))

constexpr int kBufferWord3 = 0x00020000;       // raw buffer, 32-bit data format
constexpr uint32_t kOutOfRange = 0x80000000u;  // past any num_records used here

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, static_cast<int>(bytes),
                                             kBufferWord3);
}

// Two values to bf16 in one v_cvt_pk_bf16_f32 (round to nearest even), a in
// the low half. Converting them one at a time costs two conversions plus a
// shift and an or.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt[3:0] in bits
// 3:0 and vmcnt[5:4] in bits 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0f70);
}

__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Device-only builtins are wrapped in __device__ functions: used directly in
// a __global__ template body they make the host-side instantiation fail,
// which silently drops the kernel's host stub.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, int8_t *lds, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LDS_AS void *)lds, 16, off, 0, 0, 0);
}
// 4 bytes per lane: 256 bytes of LDS per wave instruction, lane l at +4 l.
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, int8_t *lds, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LDS_AS void *)lds, 4, off, 0, 0, 0);
}
// Instruction-group ordering for the scheduler (sched_group_barrier masks:
// 0x008 MFMA, 0x100 LDS read, 0x020 global/buffer read). One MFMA, then one
// LDS read while any remain, then one buffer load while any remain, repeated:
// the fragment reads and tile loads of a K step are spread over its MFMAs.
template <int I, int NM, int NR, int ND>
__device__ __forceinline__ void interleave_from() {
    if constexpr (I < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (I < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if constexpr (I < ND) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        interleave_from<I + 1, NM, NR, ND>();
    }
}

// A no-op that mentions an AGPR. A kernel limited to 256 registers per wave
// that never names an AGPR gets its MFMAs in the VGPR form (accumulators in
// VGPRs), which measured ~20% slower here than the AGPR form: the MFMA's
// accumulator traffic then competes with the fragment reads for VGPR ports.
__device__ __forceinline__ void prefer_agpr_mfma() { asm volatile("" ::"a"(0)); }
__device__ __forceinline__ void keep_args(const void *a, const void *b, const void *c,
                                          const void *d) {
    asm volatile("" ::"s"(a), "s"(b), "s"(c), "s"(d));
}

// Workgroup barrier without a memory fence. Ordering of LDS accesses around
// it is by the explicit waits; the empty asm statements keep the compiler
// from moving memory operations across.
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

// The same products on 16 x 16 output blocks with a 64-byte K step
// (v_mfma_i32_16x16x64_i8, v_mfma_f32_16x16x32_bf16): a quarter of the
// accumulator bytes per instruction for half the multiply-adds, so half the
// accumulator traffic per multiply-add. A loop of nothing but these MFMAs on
// random operands holds a higher clock under the power limit than one of the
// 32 x 32 forms (4.15 against 2.80 POP/s for int8 in one job).
struct I8Op16 {
    using Acc = v4i;
    __device__ static Acc mma(v4i a, v4i b, Acc c) {
        return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
    }
};

typedef float v4f __attribute__((ext_vector_type(4)));
struct Bf16Op16 {
    using Acc = v4f;
    __device__ static Acc mma(v4i a, v4i b, Acc c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                       __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
    }
};

template <class Op>
struct Narrow;
template <>
struct Narrow<I8Op> {
    using type = I8Op16;
};
template <>
struct Narrow<Bf16Op> {
    using type = Bf16Op16;
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

// Epilogue of one wave: its TJ x 32 tokens starting at row mbase of the tile
// and its TI x 32 channels starting at channel nbase. In block (i, j),
// accumulator element r of lane l holds channel 32 i + 8 (r / 4) + 4 (l / 32)
// + r % 4 and token 32 j + l % 32: each quad r = 4g..4g+3 is 4 consecutive
// channels. The operands are loaded once, before the main loop.
template <int TI, int TJ, int EPI, bool N_VEC, bool HAS_BIAS>
struct Epi {
    float xs_[TJ];
    float ws_[TI][4][4];
    uint32_t b_[TI][4][2];  // bf16 pairs, converted when stored

    __device__ __forceinline__ void load(const float *xs, const float *ws, const uint16_t *bias,
                                         int m0, int rows_x, int mbase, int nbase, int N, int frow,
                                         int fhalf) {
        // Range-checked loads (zero past M / N, or for a missing bias): no
        // branch, and nothing consumes them before the epilogue.
        const __amdgpu_buffer_rsrc_t rxs =
            make_rsrc(EPI == kDequantBf16 ? xs + m0 : nullptr,
                      EPI == kDequantBf16 ? static_cast<uint32_t>(rows_x) * 4u : 0u);
        const __amdgpu_buffer_rsrc_t rws =
            make_rsrc(ws, EPI == kDequantBf16 ? static_cast<uint32_t>(N) * 4u : 0u);
        const __amdgpu_buffer_rsrc_t rbs =
            make_rsrc(bias, HAS_BIAS ? static_cast<uint32_t>(N) * 2u : 0u);
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            const uint32_t ml = mbase + 32 * j + frow;
            xs_[j] = __builtin_bit_cast(float,
                                        __builtin_amdgcn_raw_buffer_load_b32(rxs, ml * 4u, 0, 0));
        }
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t n = nbase + 32 * i + 8 * g + 4 * fhalf;
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
                        ws_[i][g][0] = ok ? w4.x : 0.0f;
                        ws_[i][g][1] = ok ? w4.y : 0.0f;
                        ws_[i][g][2] = ok ? w4.z : 0.0f;
                        ws_[i][g][3] = ok ? w4.w : 0.0f;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) ws_[i][g][e] = 0.0f;
                    }
                    b_[i][g][0] = 0u;
                    b_[i][g][1] = 0u;
                    if constexpr (HAS_BIAS) {
                        const uint2 b2 = *reinterpret_cast<const uint2 *>(bias + nc);
                        b_[i][g][0] = ok ? b2.x : 0u;
                        b_[i][g][1] = ok ? b2.y : 0u;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        ws_[i][g][e] = __builtin_bit_cast(
                            float, __builtin_amdgcn_raw_buffer_load_b32(rws, (n + e) * 4u, 0, 0));
#pragma unroll
                    for (int h = 0; h < 2; ++h)
                        b_[i][g][h] =
                            __builtin_amdgcn_raw_buffer_load_b16(rbs, (n + 2 * h) * 2u, 0, 0) |
                            static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(
                                rbs, (n + 2 * h + 1) * 2u, 0, 0))
                                << 16;
                }
            }
    }

    // The same operands from the LDS copy written by fill_lds() (tile-local
    // indices: token mbase.., channel nbase..).
    __device__ __forceinline__ void load_lds(const float *xs_l, const float *ws_l,
                                             const uint16_t *b_l, int mbase, int nbase, int frow,
                                             int fhalf) {
#pragma unroll
        for (int j = 0; j < TJ; ++j) xs_[j] = xs_l[mbase + 32 * j + frow];
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = nbase + 32 * i + 8 * g + 4 * fhalf;
                const float4 w4 = *reinterpret_cast<const float4 *>(ws_l + n);
                ws_[i][g][0] = w4.x;
                ws_[i][g][1] = w4.y;
                ws_[i][g][2] = w4.z;
                ws_[i][g][3] = w4.w;
                const uint2 b2 = *reinterpret_cast<const uint2 *>(b_l + n);
                b_[i][g][0] = b2.x;
                b_[i][g][1] = b2.y;
            }
    }

    // Writes a tile's operands to LDS (one wave): x_scale of BM tokens,
    // w_scale and bias of BN channels, zero past M / N or without a bias.
    template <int BM, int BN>
    __device__ static void fill_lds(float *xs_l, float *ws_l, uint16_t *b_l, const float *xs,
                                    const float *ws, const uint16_t *bias, int m0, int rows_x,
                                    int n0, int rows_w, int lane) {
#pragma unroll
        for (int t = lane; t < BM; t += 64)
            xs_l[t] = (EPI == kDequantBf16 && t < rows_x) ? xs[m0 + t] : 0.0f;
#pragma unroll
        for (int t = lane; t < BN; t += 64) {
            ws_l[t] = (EPI == kDequantBf16 && t < rows_w) ? ws[n0 + t] : 0.0f;
            b_l[t] = (HAS_BIAS && t < rows_w) ? bias[n0 + t] : static_cast<uint16_t>(0);
        }
    }

    template <class Acc>
    __device__ __forceinline__ void store(const Acc (&acc)[TI][TJ], void *Yout, int m0,
                                          int rows_x, int mbase, int nbase, int N, int frow,
                                          int fhalf) const {
        constexpr uint32_t kYBytes = EPI == kStoreI32 ? 4u : 2u;
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * kYBytes,
                      static_cast<uint32_t>(rows_x) * N * kYBytes);
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            const uint32_t row_off = static_cast<uint32_t>(mbase + 32 * j + frow) * N;
#pragma unroll
            for (int i = 0; i < TI; ++i) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int n = nbase + 32 * i + 8 * g + 4 * fhalf;
                    if constexpr (EPI == kStoreI32) {
                        if (N_VEC && n + 3 < N) {
                            const v4i v = {acc[i][j][4 * g], acc[i][j][4 * g + 1],
                                           acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
                            __builtin_amdgcn_raw_buffer_store_b128(v, ry, (row_off + n) * 4u, 0, 0);
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const uint32_t off =
                                    n + e < N ? (row_off + n + e) * 4u : kOutOfRange;
                                __builtin_amdgcn_raw_buffer_store_b32(acc[i][j][4 * g + e], ry, off,
                                                                      0, 0);
                            }
                        }
                    } else {
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float a = static_cast<float>(acc[i][j][4 * g + e]);
                            const uint32_t bw = b_[i][g][e >> 1];
                            const float b =
                                __uint_as_float((e & 1) ? (bw & 0xffff0000u) : (bw << 16));
                            if constexpr (EPI == kDequantBf16)
                                y[e] = __builtin_fmaf(a, xs_[j] * ws_[i][g][e], b);
                            else
                                y[e] = a + b;
                        }
                        const uint32_t p01 = f32x2_to_bf16x2(y[0], y[1]);
                        const uint32_t p23 = f32x2_to_bf16x2(y[2], y[3]);
                        const uint32_t h[4] = {p01 & 0xffffu, p01 >> 16, p23 & 0xffffu, p23 >> 16};
                        if (N_VEC && n + 3 < N) {
                            const v2u v = {p01, p23};
                            __builtin_amdgcn_raw_buffer_store_b64(v, ry, (row_off + n) * 2u, 0, 0);
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const uint32_t off =
                                    n + e < N ? (row_off + n + e) * 2u : kOutOfRange;
                                __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h[e]),
                                                                      ry, off, 0, 0);
                            }
                        }
                    }
                }
            }
        }
    }

    // The bf16 epilogues through LDS. The per-lane layout of the accumulators
    // puts the 32 lanes of an 8-byte store on 32 different output rows (64
    // cache lines per store instruction). Instead the wave writes its
    // 32 TJ x 32 TI tile of bf16 into `stage` (its own region, rows padded
    // by 16 bytes against bank conflicts), then stores whole rows: 16 bytes
    // per lane, 8 lanes per 128-byte row, 8 rows per instruction. Nothing
    // else uses `stage`, so no barrier is needed between the two passes.
    static constexpr int kRowStride = 64 * TI + 16;
    static constexpr int kStageBytes = 32 * TJ * kRowStride;

    template <class Acc>
    __device__ __forceinline__ void store_rows(const Acc (&acc)[TI][TJ], int8_t *stage,
                                               void *Yout, int m0, int rows_x, int mbase,
                                               int nbase, int N, int frow, int fhalf,
                                               int lane) const {
        static_assert(EPI != kStoreI32, "row stores are for the bf16 epilogues");
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    float y[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float a = static_cast<float>(acc[i][j][4 * g + e]);
                        const uint32_t bw = b_[i][g][e >> 1];
                        const float b = __uint_as_float((e & 1) ? (bw & 0xffff0000u) : (bw << 16));
                        if constexpr (EPI == kDequantBf16)
                            y[e] = __builtin_fmaf(a, xs_[j] * ws_[i][g][e], b);
                        else
                            y[e] = a + b;
                    }
                    const int t = 32 * j + frow;
                    const int c = 32 * i + 8 * g + 4 * fhalf;
                    *reinterpret_cast<v2u *>(stage + t * kRowStride + c * 2) =
                        v2u{f32x2_to_bf16x2(y[0], y[1]), f32x2_to_bf16x2(y[2], y[3])};
                }
        constexpr int CPR = 64 * TI / 16;  // 16-byte chunks per row
        constexpr int ROUNDS = 32 * TJ * CPR / 64;
        static_assert(32 * TJ * CPR % 64 == 0, "whole store rounds");
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * 2,
                      static_cast<uint32_t>(rows_x) * N * 2u);
        const bool vec8 = (N & 7) == 0;
#pragma unroll
        for (int r = 0; r < ROUNDS; ++r) {
            const int id = r * 64 + lane;
            const int row = id / CPR;
            const int c = id % CPR;
            const v4i v = *reinterpret_cast<const v4i *>(stage + row * kRowStride + c * 16);
            const int n = nbase + 8 * c;
            const uint32_t base = static_cast<uint32_t>(mbase + row) * N;
            if (vec8 && n + 8 <= N) {
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, (base + n) * 2u, 0, 0);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t off = n + e < N ? (base + n + e) * 2u : kOutOfRange;
                    __builtin_amdgcn_raw_buffer_store_b16(
                        static_cast<uint16_t>(static_cast<uint32_t>(v[e >> 1]) >> (16 * (e & 1))),
                        ry, off, 0, 0);
                }
            }
        }
    }

    // store_slices with the operands read from their LDS copy as each
    // group of four channels is converted (tile-local token mbase.., channel
    // nbase..; n0 is the tile's first channel), not held in registers for
    // the whole epilogue. N % 8 == 0.
    template <class Acc>
    __device__ __forceinline__ void store_slices_lds(const Acc (&acc)[TI][TJ], int8_t *stage,
                                                     const float *xs_l, const float *ws_l,
                                                     const uint16_t *b_l, void *Yout, int m0,
                                                     int rows_x, int mbase, int nbase, int n0,
                                                     int N, int frow, int fhalf, int lane) const {
        static_assert(EPI != kStoreI32, "row stores are for the bf16 epilogues");
        constexpr int CPR = 64 * TI / 16;  // 16-byte chunks per row
        constexpr int ROUNDS = 32 * CPR / 64;
        static_assert(32 * CPR % 64 == 0, "whole store rounds");
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * 2,
                      static_cast<uint32_t>(rows_x) * N * 2u);
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            const float xv = EPI == kDequantBf16 ? xs_l[mbase + 32 * j + frow] : 0.0f;
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c = 32 * i + 8 * g + 4 * fhalf;
                    float4 w4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                    if constexpr (EPI == kDequantBf16)
                        w4 = *reinterpret_cast<const float4 *>(ws_l + nbase + c);
                    uint2 b2 = make_uint2(0u, 0u);
                    if constexpr (HAS_BIAS) b2 = *reinterpret_cast<const uint2 *>(b_l + nbase + c);
                    const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
                    const uint32_t bw[2] = {b2.x, b2.y};
                    float y[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float a = static_cast<float>(acc[i][j][4 * g + e]);
                        const float b =
                            __uint_as_float((e & 1) ? (bw[e >> 1] & 0xffff0000u) : (bw[e >> 1] << 16));
                        if constexpr (EPI == kDequantBf16)
                            y[e] = __builtin_fmaf(a, xv * wv[e], b);
                        else
                            y[e] = a + b;
                    }
                    *reinterpret_cast<v2u *>(stage + frow * kRowStride + c * 2) =
                        v2u{f32x2_to_bf16x2(y[0], y[1]), f32x2_to_bf16x2(y[2], y[3])};
                }
#pragma unroll
            for (int r = 0; r < ROUNDS; ++r) {
                const int id = r * 64 + lane;
                const int row = id / CPR;
                const int c = id % CPR;
                const v4i v = *reinterpret_cast<const v4i *>(stage + row * kRowStride + c * 16);
                const int n = n0 + nbase + 8 * c;
                const uint32_t base = static_cast<uint32_t>(mbase + 32 * j + row) * N;
                const uint32_t off = n + 8 <= N ? (base + n) * 2u : kOutOfRange;
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, off, 0, 0);
            }
        }
    }

    // store_rows one 32-token slice at a time, for workgroups whose LDS
    // cannot stage every wave's whole tile: `stage` holds kSliceBytes.
    static constexpr int kSliceBytes = 32 * kRowStride;

    template <class Acc>
    __device__ __forceinline__ void store_slices(const Acc (&acc)[TI][TJ], int8_t *stage,
                                                 void *Yout, int m0, int rows_x, int mbase,
                                                 int nbase, int N, int frow, int fhalf,
                                                 int lane) const {
        static_assert(EPI != kStoreI32, "row stores are for the bf16 epilogues");
        constexpr int CPR = 64 * TI / 16;  // 16-byte chunks per row
        constexpr int ROUNDS = 32 * CPR / 64;
        static_assert(32 * CPR % 64 == 0, "whole store rounds");
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * 2,
                      static_cast<uint32_t>(rows_x) * N * 2u);
        const bool vec8 = (N & 7) == 0;
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
            // A wave's LDS accesses execute in order: the reads of slice j - 1
            // below are done before these writes replace it.
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    float y[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float a = static_cast<float>(acc[i][j][4 * g + e]);
                        const uint32_t bw = b_[i][g][e >> 1];
                        const float b =
                            __uint_as_float((e & 1) ? (bw & 0xffff0000u) : (bw << 16));
                        if constexpr (EPI == kDequantBf16)
                            y[e] = __builtin_fmaf(a, xs_[j] * ws_[i][g][e], b);
                        else
                            y[e] = a + b;
                    }
                    const int c = 32 * i + 8 * g + 4 * fhalf;
                    *reinterpret_cast<v2u *>(stage + frow * kRowStride + c * 2) =
                        v2u{f32x2_to_bf16x2(y[0], y[1]), f32x2_to_bf16x2(y[2], y[3])};
                }
#pragma unroll
            for (int r = 0; r < ROUNDS; ++r) {
                const int id = r * 64 + lane;
                const int row = id / CPR;
                const int c = id % CPR;
                const v4i v = *reinterpret_cast<const v4i *>(stage + row * kRowStride + c * 16);
                const int n = nbase + 8 * c;
                const uint32_t base = static_cast<uint32_t>(mbase + 32 * j + row) * N;
                if (vec8 && n + 8 <= N) {
                    __builtin_amdgcn_raw_buffer_store_b128(v, ry, (base + n) * 2u, 0, 0);
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t off = n + e < N ? (base + n + e) * 2u : kOutOfRange;
                        __builtin_amdgcn_raw_buffer_store_b16(
                            static_cast<uint16_t>(static_cast<uint32_t>(v[e >> 1]) >>
                                                  (16 * (e & 1))),
                            ry, off, 0, 0);
                    }
                }
            }
        }
    }
};

// MFMA side of one wave: fragment reads from an LDS slot and the MFMAs of a
// WTN x WTM wave tile (TI channel blocks, TJ token blocks). Lane l reads row
// l % 32 of a 32-row block, chunk 2 s + l / 32 of the K tile; the swizzle key
// depends on l only.
template <class Op, int BM, int BK, int TI, int TJ, int SWZ>
struct Mma {
    static constexpr int CPR = BK / 16;
    typename Op::Acc acc[TI][TJ];
    v4i wf[2][TI];
    v4i xf[2][TJ];
    int x_base, w_base, fhalf, fkey;

    __device__ __forceinline__ void init(int lane, int mbase, int nbase) {
        const int frow = lane & 31;
        fhalf = lane >> 5;
        fkey = (frow >> SWZ) & (CPR - 1);
        x_base = (mbase + frow) * BK;
        w_base = BM * BK + (nbase + frow) * BK;
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int j = 0; j < TJ; ++j) acc[i][j] = typename Op::Acc{};
    }
    __device__ __forceinline__ void load(const int8_t *slot, int s, int buf) {
        const int chunk = (2 * s + fhalf) ^ fkey;
#pragma unroll
        for (int i = 0; i < TI; ++i)
            wf[buf][i] = *reinterpret_cast<const v4i *>(slot + w_base + i * 32 * BK + chunk * 16);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
            xf[buf][j] = *reinterpret_cast<const v4i *>(slot + x_base + j * 32 * BK + chunk * 16);
    }
    // X fragment outer, W fragments alternating (as in Mma16::half).
    __device__ __forceinline__ void step(int buf) {
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int ii = 0; ii < TI; ++ii) {
                const int i = (j & 1) ? TI - 1 - ii : ii;
                acc[i][j] = Op::mma(wf[buf][i], xf[buf][j], acc[i][j]);
            }
    }
    // One K tile whose data is in `slot`. Steps 0..KSTEPS-2 read the next
    // step's fragments, then run the current MFMAs. Before the last step
    // comes `boundary()` (the tile hand-over, see the kernels) unless this is
    // the last tile; it ends by reading the next tile's first fragments.
    // Scheduling barriers keep each group of reads ahead of the MFMAs it
    // overlaps (the compiler would otherwise sink the reads to their uses).
    template <bool LAST, class Boundary>
    __device__ __forceinline__ void tile(const int8_t *slot, Boundary &&boundary) {
        constexpr int KSTEPS = BK / 32;
        static_assert(KSTEPS % 2 == 0, "fragment buffer 0 starts every tile");
#pragma unroll
        for (int s = 0; s + 1 < KSTEPS; ++s) {
            load(slot, s + 1, (s + 1) & 1);
            sched_fence();
            step(s & 1);
            sched_fence();
        }
        if constexpr (!LAST) {
            boundary();
            sched_fence();
        }
        step((KSTEPS - 1) & 1);
        sched_fence();
    }
};

// MFMA side of one wave of gemm_2s_kernel: like Mma, with separate X and W
// slots and fragments read two MFMA steps ahead, one register buffer per
// step of the 4-step (128-byte) K tile. A wave running alone on its SIMD
// (the other one waiting at the barrier) then still has two steps of MFMAs
// to cover each LDS read.
template <class Op, int BK, int TI, int TJ, int SWZ>
struct Mma2 {
    static constexpr int CPR = BK / 16;
    static constexpr int KSTEPS = BK / 32;
    static_assert(KSTEPS == 4, "four MFMA steps per K tile");
    typename Op::Acc acc[TI][TJ];
    v4i wf[KSTEPS][TI];
    v4i xf[KSTEPS][TJ];
    int x_row, w_row, fhalf, fkey;

    __device__ __forceinline__ void init(int lane, int mbase, int nbase) {
        const int frow = lane & 31;
        fhalf = lane >> 5;
        fkey = (frow >> SWZ) & (CPR - 1);
        x_row = (mbase + frow) * BK;
        w_row = (nbase + frow) * BK;
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int j = 0; j < TJ; ++j) acc[i][j] = typename Op::Acc{};
    }
    // Fragments of MFMA step s (0..3) of a K tile into buffer s.
    template <int S>
    __device__ __forceinline__ void load(const int8_t *xslot, const int8_t *wslot) {
        const int chunk = (2 * S + fhalf) ^ fkey;
#pragma unroll
        for (int i = 0; i < TI; ++i)
            wf[S][i] = *reinterpret_cast<const v4i *>(wslot + w_row + i * 32 * BK + chunk * 16);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
            xf[S][j] = *reinterpret_cast<const v4i *>(xslot + x_row + j * 32 * BK + chunk * 16);
    }
    // X fragment outer, W fragments in alternating order, as in Mma16::half
    // (here 0.1-0.4% faster than W outer at three 192 x 256 shapes, outputs
    // identical).
    template <int S>
    __device__ __forceinline__ void step() {
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int ii = 0; ii < TI; ++ii) {
                const int i = (j & 1) ? TI - 1 - ii : ii;
                acc[i][j] = Op::mma(wf[S][i], xf[S][j], acc[i][j]);
            }
    }
    // One K tile. On entry buffers 0 and 1 hold its steps 0 and 1. Steps 0
    // and 1 read steps 2 and 3; then `boundary()`; then, unless LAST, steps
    // 2 and 3 read steps 0 and 1 of the next tile from (nxslot, nwslot), and
    // LOADS loads (`issue(i)`) go out during step 2.
    template <bool LAST, int LOADS, class Boundary, class Issue>
    __device__ __forceinline__ void tile(const int8_t *xslot, const int8_t *wslot,
                                         const int8_t *nxslot, const int8_t *nwslot,
                                         Boundary &&boundary, Issue &&issue) {
        load<2>(xslot, wslot);
        step<0>();
        interleave_from<0, TI * TJ, TI + TJ, 0>();
        sched_fence();
        load<3>(xslot, wslot);
        step<1>();
        interleave_from<0, TI * TJ, TI + TJ, 0>();
        sched_fence();
        if constexpr (!LAST) {
            boundary();
            sched_fence();
#pragma unroll
            for (int i = 0; i < LOADS; ++i) issue(i);
            load<0>(nxslot, nwslot);
        }
        step<2>();
        interleave_from<0, TI * TJ, LAST ? 0 : TI + TJ, LOADS>();
        sched_fence();
        if constexpr (!LAST) load<1>(nxslot, nwslot);
        step<3>();
        interleave_from<0, TI * TJ, LAST ? 0 : TI + TJ, 0>();
        sched_fence();
    }
};

// Epilogue of one wave for the 16 x 16 blocks of Mma16. In block (i, a, j, b)
// element e of lane l holds channel 32 i + 16 a + 4 (l / 16) + e and token
// 32 j + 16 b + l % 16 of the wave's tile: each accumulator is 4
// consecutive channels of one token.
template <int TI, int TJ, int EPI, bool N_VEC, bool HAS_BIAS>
struct Epi16 {
    static constexpr int kRowStride = 64 * TI + 16;
    static constexpr int kSliceBytes = 32 * kRowStride;

    // int32 accumulators straight to C (nbase: the wave's first channel in
    // the whole output). Rows past M fall outside the resource; channels past
    // N are not stored. N_VEC: N % 4 == 0, so 4 channels go out as one
    // aligned 16-byte store.
    template <class Acc>
    __device__ __forceinline__ void store(const Acc (&acc)[TI][2][TJ][2], void *Yout, int m0,
                                          int rows_x, int mbase, int nbase, int N,
                                          int lane) const {
        static_assert(EPI == kStoreI32, "the int32 store");
        const int r16 = lane & 15, kg = lane >> 4;
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * 4,
                      static_cast<uint32_t>(rows_x) * N * 4u);
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const uint32_t row_off = static_cast<uint32_t>(mbase + 32 * j + 16 * b + r16) * N;
#pragma unroll
                for (int i = 0; i < TI; ++i)
#pragma unroll
                    for (int a = 0; a < 2; ++a) {
                        const int n = nbase + 32 * i + 16 * a + 4 * kg;
                        if (N_VEC && n + 3 < N) {
                            __builtin_amdgcn_raw_buffer_store_b128(acc[i][a][j][b], ry,
                                                                   (row_off + n) * 4u, 0, 0);
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const uint32_t off =
                                    n + e < N ? (row_off + n + e) * 4u : kOutOfRange;
                                __builtin_amdgcn_raw_buffer_store_b32(acc[i][a][j][b][e], ry, off,
                                                                      0, 0);
                            }
                        }
                    }
            }
    }

    // The bf16 epilogues, one 32-token slice at a time through `stage`
    // (kSliceBytes of the wave's own), with the operands read from their LDS
    // copy (tile-local token mbase.., channel nbase..; n0 is the tile's first
    // channel). Each slice is converted into `stage` as 4-channel groups,
    // then stored as whole rows: 16 bytes per lane, 8 lanes per 128-byte row.
    // A wave's LDS accesses execute in order, so the row reads of slice j - 1
    // are done before slice j is written over them. The operand copies hold
    // zeros past N; where N % 8 != 0 the rows go out element by element.
    template <class Acc>
    __device__ __forceinline__ void store_slices_lds(const Acc (&acc)[TI][2][TJ][2],
                                                     int8_t *stage, const float *xs_l,
                                                     const float *ws_l, const uint16_t *b_l,
                                                     void *Yout, int m0, int rows_x, int mbase,
                                                     int nbase, int n0, int N, int lane) const {
        static_assert(EPI != kStoreI32, "row stores are for the bf16 epilogues");
        constexpr int CPR = 64 * TI / 16;  // 16-byte chunks per row
        constexpr int ROUNDS = 32 * CPR / 64;
        static_assert(32 * CPR % 64 == 0, "whole store rounds");
        const int r16 = lane & 15, kg = lane >> 4;
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(static_cast<int8_t *>(Yout) + static_cast<int64_t>(m0) * N * 2,
                      static_cast<uint32_t>(rows_x) * N * 2u);
        const bool vec8 = (N & 7) == 0;
#pragma unroll
        for (int j = 0; j < TJ; ++j) {
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int t = 16 * b + r16;
                const float xv = EPI == kDequantBf16 ? xs_l[mbase + 32 * j + t] : 0.0f;
#pragma unroll
                for (int i = 0; i < TI; ++i)
#pragma unroll
                    for (int a = 0; a < 2; ++a) {
                        const int c = 32 * i + 16 * a + 4 * kg;
                        float4 w4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                        if constexpr (EPI == kDequantBf16)
                            w4 = *reinterpret_cast<const float4 *>(ws_l + nbase + c);
                        uint2 b2 = make_uint2(0u, 0u);
                        if constexpr (HAS_BIAS)
                            b2 = *reinterpret_cast<const uint2 *>(b_l + nbase + c);
                        const float wv[4] = {w4.x, w4.y, w4.z, w4.w};
                        const uint32_t bw[2] = {b2.x, b2.y};
                        float y[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float v = static_cast<float>(acc[i][a][j][b][e]);
                            const float bb = __uint_as_float((e & 1) ? (bw[e >> 1] & 0xffff0000u)
                                                                     : (bw[e >> 1] << 16));
                            if constexpr (EPI == kDequantBf16)
                                y[e] = __builtin_fmaf(v, xv * wv[e], bb);
                            else
                                y[e] = v + bb;
                        }
                        *reinterpret_cast<v2u *>(stage + t * kRowStride + c * 2) =
                            v2u{f32x2_to_bf16x2(y[0], y[1]), f32x2_to_bf16x2(y[2], y[3])};
                    }
            }
#pragma unroll
            for (int r = 0; r < ROUNDS; ++r) {
                const int id = r * 64 + lane;
                const int row = id / CPR;
                const int c = id % CPR;
                const v4i v = *reinterpret_cast<const v4i *>(stage + row * kRowStride + c * 16);
                const int n = n0 + nbase + 8 * c;
                const uint32_t base = static_cast<uint32_t>(mbase + 32 * j + row) * N;
                if (vec8 || n + 8 <= N) {
                    const uint32_t off = n + 8 <= N ? (base + n) * 2u : kOutOfRange;
                    __builtin_amdgcn_raw_buffer_store_b128(v, ry, off, 0, 0);
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const uint32_t off = n + e < N ? (base + n + e) * 2u : kOutOfRange;
                        __builtin_amdgcn_raw_buffer_store_b16(
                            static_cast<uint16_t>(static_cast<uint32_t>(v[e >> 1]) >>
                                                  (16 * (e & 1))),
                            ry, off, 0, 0);
                    }
                }
            }
        }
    }
};

// MFMA side of one wave of gemm_pt_kernel with the 16 x 16 x 64-byte MFMAs:
// TI x TJ blocks of 32 x 32 (channels x tokens), each 2 x 2 MFMA blocks
// acc[i][a][j][b] (channels 32 i + 16 a.., tokens 32 j + 16 b..). Lane l
// reads row l % 16 of a 16-row block, chunk 4 s + l / 16 of the K tile's
// 64-byte step s; the swizzle key depends on l only, since every block
// starts on a multiple of 16 rows. Each step runs as two halves, one per
// token half b, and the fragments are read one half ahead: the W fragments
// of a step (2 TI) serve both halves, the X fragments (TJ) one half. At
// most two steps' W fragments and two halves' X fragments are live (56
// registers for TI = 2, TJ = 3), which the 168 registers of a wave at
// three waves per SIMD hold.
template <class Op, int BK, int TI, int TJ, int SWZ>
struct Mma16 {
    static constexpr int CPR = BK / 16;
    static_assert(BK == 128, "two 64-byte MFMA steps per K tile");
    typename Op::Acc acc[TI][2][TJ][2];
    v4i wf[2][TI][2];  // by step parity
    v4i xf[2][TJ];     // by token half
    int x_off[2], w_off[2];  // the lane's row and swizzled chunk, per step

    __device__ __forceinline__ void init(int lane, int mbase, int nbase) {
        const int r16 = lane & 15;
        const int kg = lane >> 4;
        const int key = (r16 >> SWZ) & (CPR - 1);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int chunk = (4 * s + kg) ^ key;
            x_off[s] = (mbase + r16) * BK + chunk * 16;
            w_off[s] = (nbase + r16) * BK + chunk * 16;
        }
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int j = 0; j < TJ; ++j)
#pragma unroll
                    for (int b = 0; b < 2; ++b) acc[i][a][j][b] = typename Op::Acc{};
    }
    template <int S, int P>
    __device__ __forceinline__ void load_w(const int8_t *wslot) {
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
            for (int a = 0; a < 2; ++a)
                wf[P][i][a] = *reinterpret_cast<const v4i *>(wslot + w_off[S] +
                                                             (32 * i + 16 * a) * BK);
    }
    template <int S, int B>
    __device__ __forceinline__ void load_x(const int8_t *xslot) {
#pragma unroll
        for (int j = 0; j < TJ; ++j)
            xf[B][j] = *reinterpret_cast<const v4i *>(xslot + x_off[S] + (32 * j + 16 * B) * BK);
    }
    // The fragments that start a K tile: step 0's W and its first token half.
    template <int S>
    __device__ __forceinline__ void load(const int8_t *xslot, const int8_t *wslot) {
        static_assert(S == 0, "a K tile starts at step 0");
        load_w<0, 0>(wslot);
        load_x<0, 0>(xslot);
    }
    // The MFMAs of token half B with the W fragments of parity P: X fragment
    // outer, W fragments in alternating order, so that consecutive MFMAs
    // share an operand, also from one X fragment to the next. Fewer operand
    // bits then change between them, and under this load the clock is set
    // by power (with the 32 x 32 blocks: 0.5-1.5% faster than W outer at the
    // DiT shapes in one job, outputs identical).
    template <int P, int B>
    __device__ __forceinline__ void half() {
#pragma unroll
        for (int j = 0; j < TJ; ++j)
#pragma unroll
            for (int ii = 0; ii < 2 * TI; ++ii) {
                const int w = (j & 1) ? 2 * TI - 1 - ii : ii;
                const int i = w >> 1, a = w & 1;
                acc[i][a][j][B] = Op::mma(wf[P][i][a], xf[B][j], acc[i][a][j][B]);
            }
    }
    // One K tile. On entry wf[0] and xf[0] hold step 0's W and first token
    // half. Halves (0,0), (0,1) and (1,0) read the next half's fragments;
    // then `boundary()`; then, unless LAST, half (1,1) reads the next tile's
    // first fragments from (nxslot, nwslot) and LOADS loads (`issue(i)`) go
    // out during it.
    template <bool LAST, int LOADS, class Boundary, class Issue>
    __device__ __forceinline__ void tile(const int8_t *xslot, const int8_t *wslot,
                                         const int8_t *nxslot, const int8_t *nwslot,
                                         Boundary &&boundary, Issue &&issue) {
        constexpr int NM = 2 * TI * TJ;  // MFMAs per half
        load_x<0, 1>(xslot);
        half<0, 0>();
        interleave_from<0, NM, TJ, 0>();
        sched_fence();
        load_w<1, 1>(wslot);
        load_x<1, 0>(xslot);
        half<0, 1>();
        interleave_from<0, NM, 2 * TI + TJ, 0>();
        sched_fence();
        load_x<1, 1>(xslot);
        half<1, 0>();
        interleave_from<0, NM, TJ, 0>();
        sched_fence();
        if constexpr (!LAST) {
            boundary();
            sched_fence();
#pragma unroll
            for (int i = 0; i < LOADS; ++i) issue(i);
            load_w<0, 0>(nwslot);
            load_x<0, 0>(nxslot);
        }
        half<1, 1>();
        interleave_from<0, NM, LAST ? 0 : 2 * TI + TJ, LOADS>();
        sched_fence();
    }
};

// Lane l of 1 KiB DMA block `blk` of a BK-wide tile writes LDS bytes
// [blk*1024 + 16 l, +16) = row blk*(1024/BK) + l / CPR, physical chunk
// l % CPR, which holds logical chunk (l % CPR) ^ swizzle(row). Returns the
// lane's source offset within the panel at K tile 0.
template <int BK, int SWZ>
__device__ __forceinline__ uint32_t dma_offset(int blk, int lane, int Kb) {
    constexpr int CPR = BK / 16;
    const int row = blk * (1024 / BK) + lane / CPR;
    const int chunk = (lane % CPR) ^ ((row >> SWZ) & (CPR - 1));
    return static_cast<uint32_t>(row) * Kb + chunk * 16;
}

// --------------------------------------------------------------------------
// gemm_kernel: every wave loads and multiplies.
// --------------------------------------------------------------------------
template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int SWZ,
          int GROUP_M, int EPI, bool N_VEC, bool HAS_BIAS>
__global__ __launch_bounds__(WAVES_M *WAVES_N * 64) void gemm_kernel(
    const int8_t *__restrict__ X, const int8_t *__restrict__ W, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int WTM = BM / WAVES_M;  // tokens per wave
    constexpr int WTN = BN / WAVES_N;  // channels per wave
    constexpr int TJ = WTM / 32;
    constexpr int TI = WTN / 32;
    constexpr int LA = BM * BK / 1024 / NW;  // 1 KiB DMA blocks per wave, X tile
    constexpr int LB = BN * BK / 1024 / NW;  // ... W tile
    constexpr int LOADS = LA + LB;
    constexpr int STAGE = (BM + BN) * BK;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(LA * NW * 1024 == BM * BK && LB * NW * 1024 == BN * BK, "DMA split");
    static_assert(BK == 64 || BK == 128, "K tile of 64 or 128 bytes");
    static_assert(STAGES >= 2 && LOADS * (STAGES - 2) < 64, "vmcnt range");
    static_assert(STAGES * STAGE <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) int8_t smem[STAGES * STAGE];

    // Materialize the epilogue's pointer arguments now: a scalar load of a
    // kernel argument left pending into the main loop would make every LDS
    // wait there a full lgkmcnt(0) (scalar loads complete out of order).
    keep_args(xs, ws, bias, Yout);

    int tm, tn;
    map_tile<GROUP_M>(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int mbase = (wave / WAVES_N) * WTM;
    const int nbase = (wave % WAVES_N) * WTN;
    const int rows_x = min(BM, M - m0);
    const int rows_w = min(BN, N - n0);

    // Epilogue operands first, and kept older than every tile load: the vmcnt
    // waits below count only tile loads as younger. (They are global loads
    // and the tile loads write LDS, so nothing else orders them.)
    Epi<TI, TJ, EPI, N_VEC, HAS_BIAS> epi;
    epi.load(xs, ws, bias, m0, rows_x, mbase, n0 + nbase, N, lane & 31, lane >> 5);
    sched_fence();

    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(X + static_cast<int64_t>(m0) * Kb, static_cast<uint32_t>(rows_x) * Kb);
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(W + static_cast<int64_t>(n0) * Kb, static_cast<uint32_t>(rows_w) * Kb);
    uint32_t off_x[LA], off_w[LB];
#pragma unroll
    for (int i = 0; i < LA; ++i) off_x[i] = dma_offset<BK, SWZ>(wave + i * NW, lane, Kb);
#pragma unroll
    for (int i = 0; i < LB; ++i) off_w[i] = dma_offset<BK, SWZ>(wave + i * NW, lane, Kb);

    const int KT = Kb / BK;  // the launcher guarantees BK divides Kb
    auto issue = [&](int kt) {
        int8_t *slot = smem + (kt % STAGES) * STAGE;
        const int kb = kt * BK;
#pragma unroll
        for (int i = 0; i < LA; ++i) dma16(rx, slot + (wave + i * NW) * 1024, off_x[i] + kb);
#pragma unroll
        for (int i = 0; i < LB; ++i)
            dma16(rw, slot + BM * BK + (wave + i * NW) * 1024, off_w[i] + kb);
    };

    Mma<Op, BM, BK, TI, TJ, SWZ> mma;
    mma.init(lane, mbase, nbase);

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
    mma.load(smem, 0, 0);

    // Tile boundary kt -> kt+1: every read of tile kt has completed (the last
    // ones were issued a whole MFMA step ago); once this wave's loads of tile
    // kt+1 are in and all waves meet, slot kt is refilled with tile
    // kt+STAGES and tile kt+1's first fragments are read. The three loops are
    // branch-free so that the compiler's own waits stay exact.
    int kt = 0;
    for (; kt + STAGES < KT; ++kt)  // refill as we go
        mma.template tile<false>(smem + (kt % STAGES) * STAGE, [&] {
            wait_lgkmcnt0();
            wait_vmcnt<LOADS * (STAGES - 2)>();
            barrier();
            issue(kt + STAGES);
            mma.load(smem + ((kt + 1) % STAGES) * STAGE, 0, 0);
        });
    for (; kt + 1 < KT; ++kt)  // drain the ring
        mma.template tile<false>(smem + (kt % STAGES) * STAGE, [&] {
            wait_lgkmcnt0();
            wait_vmcnt<0>();
            barrier();
            mma.load(smem + ((kt + 1) % STAGES) * STAGE, 0, 0);
        });
    mma.template tile<true>(smem + (kt % STAGES) * STAGE, [] {});

    epi.store(mma.acc, Yout, m0, rows_x, mbase, n0 + nbase, N, lane & 31, lane >> 5);
}

// --------------------------------------------------------------------------
// gemm_2s_kernel: four loading waves, two-slot rings. Made for large tiles
// (192 x 256: 27% fewer bytes per MFMA than 256 x 128; 288 x 256 with 12
// waves: 19% fewer than 192 x 256) whose accumulators leave no registers
// for separate producer waves. One barrier per K tile, placed once every
// fragment read of the tile has been issued: before its third MFMA step
// when fragments are read two steps ahead (8 waves), before its fourth when
// one step ahead (12 waves):
//   barrier #kt+1: every wave has finished reading the slots of tile kt and
//   its own loads of tile kt+1 have landed.
// Right after it each wave issues its share of tile kt+2 into the slots
// just freed, so a tile's loads have most of a K tile of MFMAs to land in.
// The epilogue operands are staged in LDS by wave 0 before barrier #0; the
// output rows go out through LDS (store_rows / store_slices), staged in the
// ring.
// --------------------------------------------------------------------------
template <class Op, int BM, int BN, int WAVES_M, int WAVES_N, int SWZ, int GROUP_M, int EPI,
          bool N_VEC, bool HAS_BIAS>
__global__ __launch_bounds__(WAVES_M *WAVES_N * 64) void gemm_2s_kernel(
    const int8_t *__restrict__ X, const int8_t *__restrict__ W, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int BK = 128;
    constexpr int NW = WAVES_M * WAVES_N;
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int TJ = WTM / 32;
    constexpr int TI = WTN / 32;
    constexpr int NBX = BM * BK / 1024;
    constexpr int NBW = BN * BK / 1024;
    // Waves 0..NI-1 load; a workgroup's waves go round-robin to the 4 SIMDs,
    // so each SIMD has one loading wave and one or two that only multiply
    // (whose MFMAs keep going while a load instruction waits to issue).
    constexpr int NI = 4;
    static_assert(NW == 8 || NW == 12, "two or three waves per SIMD");
    constexpr int LX = NBX / NI;  // 1 KiB DMA blocks per loading wave and K tile, X
    constexpr int LW = NBW / NI;  // ... W
    constexpr int XSLOT = BM * BK;
    constexpr int WSLOT = BN * BK;
    constexpr int RING = 2 * (XSLOT + WSLOT);
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(LX * NI == NBX && LW * NI == NBW, "DMA split");
    static_assert(LX + LW < 64, "vmcnt range");

    using EpiT = Epi<TI, TJ, EPI, N_VEC, HAS_BIAS>;
    // The ring; after the last K tile the same bytes stage the waves' output
    // rows (whole wave tiles if they fit, else 32-token slices). Then the
    // epilogue operands.
    constexpr bool SLICED = NW * EpiT::kStageBytes > RING;
    constexpr int STAGE_BYTES = SLICED ? EpiT::kSliceBytes : EpiT::kStageBytes;
    constexpr int BODY = RING > NW * STAGE_BYTES ? RING : NW * STAGE_BYTES;
    static_assert(BODY + 4 * BM + 6 * BN <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) int8_t smem[BODY + 4 * BM + 6 * BN];
    int8_t *xring = smem;
    int8_t *wring = smem + 2 * XSLOT;
    float *ep_xs = reinterpret_cast<float *>(smem + BODY);
    float *ep_ws = ep_xs + BM;
    uint16_t *ep_b = reinterpret_cast<uint16_t *>(ep_ws + BN);
    keep_args(xs, ws, bias, Yout);

    int tm, tn;
    map_tile<GROUP_M>(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int mbase = (wave / WAVES_N) * WTM;
    const int nbase = (wave % WAVES_N) * WTN;
    const int rows_x = min(BM, M - m0);
    const int rows_w = min(BN, N - n0);
    const int KT = Kb / BK;  // the launcher guarantees BK divides Kb

    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(X + static_cast<int64_t>(m0) * Kb, static_cast<uint32_t>(rows_x) * Kb);
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(W + static_cast<int64_t>(n0) * Kb, static_cast<uint32_t>(rows_w) * Kb);
    const bool loader = wave < NI;
    const int iw = loader ? wave : 0;  // index among the loading waves
    uint32_t off_x[LX], off_w[LW];
#pragma unroll
    for (int i = 0; i < LX; ++i) off_x[i] = dma_offset<BK, SWZ>(iw + i * NI, lane, Kb);
#pragma unroll
    for (int i = 0; i < LW; ++i) off_w[i] = dma_offset<BK, SWZ>(iw + i * NI, lane, Kb);
    auto xslot = [&](int kt) { return xring + (kt & 1) * XSLOT; };
    auto wslot = [&](int kt) { return wring + (kt & 1) * WSLOT; };
    // Load i of this wave's share of tile kt: W blocks first, then X blocks.
    auto issue_one = [&](int kt, int i) {
        if (!loader) return;
        if (i < LW)
            dma16(rw, wslot(kt) + (iw + i * NI) * 1024, off_w[i] + kt * BK);
        else
            dma16(rx, xslot(kt) + (iw + (i - LW) * NI) * 1024, off_x[i - LW] + kt * BK);
    };

    // Fragments two MFMA steps ahead at two waves per SIMD (32 x 32 blocks);
    // at three, the 16 x 16 blocks of Mma16, read one half step ahead.
    constexpr bool AHEAD2 = NW == 8;
    std::conditional_t<AHEAD2, Mma2<Op, BK, TI, TJ, SWZ>,
                       Mma16<typename Narrow<Op>::type, BK, TI, TJ, SWZ>>
        mma;
    // Accumulators in AGPRs at two waves per SIMD. At three, a wave has 168
    // registers, which the compiler splits evenly between VGPRs and AGPRs
    // once a kernel uses AGPRs: 96 accumulators in 84 AGPRs spill. In the
    // VGPR form of the MFMAs everything fits in 165 VGPRs.
    if constexpr (AHEAD2) prefer_agpr_mfma();
    mma.init(lane, mbase, nbase);

#pragma unroll
    for (int i = 0; i < LW + LX; ++i) issue_one(0, i);
    if (EPI != kStoreI32 && wave == 0)
        EpiT::template fill_lds<BM, BN>(ep_xs, ep_ws, ep_b, xs, ws, bias, m0, rows_x, n0,
                                        rows_w, lane);
    wait_vmcnt<0>();
    wait_lgkmcnt0();
    barrier();  // #0
    if (KT > 1) {
#pragma unroll
        for (int i = 0; i < LW + LX; ++i) issue_one(1, i);
    }
    mma.template load<0>(xslot(0), wslot(0));
    if constexpr (AHEAD2) mma.template load<1>(xslot(0), wslot(0));

    // Tile kt's loads went out at barrier #kt-1 (tiles 0 and 1 in the
    // prologue). Branch-free loops keep the compiler's own waits exact.
    auto boundary = [&] {
        wait_lgkmcnt0();  // this wave's reads of tile kt's slots are done
        wait_vmcnt<0>();  // and its loads of tile kt+1 have landed
        barrier();        // #kt+1
    };
    int kt = 0;
    auto issue_kt2 = [&](int i) { issue_one(kt + 2, i); };
    for (; kt + 2 < KT; ++kt)
        mma.template tile<false, LW + LX>(xslot(kt), wslot(kt), xslot(kt + 1), wslot(kt + 1),
                                          boundary, issue_kt2);
    if (kt + 1 < KT) {
        mma.template tile<false, 0>(xslot(kt), wslot(kt), xslot(kt + 1), wslot(kt + 1),
                                    boundary, [](int) {});
        ++kt;
    }
    mma.template tile<true, 0>(xslot(kt), wslot(kt), xslot(kt), wslot(kt), [] {}, [](int) {});

    if constexpr (!AHEAD2) {
        Epi16<TI, TJ, EPI, N_VEC, HAS_BIAS> epi;
        static_assert(SLICED, "12 waves stage 32-token slices");
        if constexpr (EPI == kStoreI32) {
            epi.store(mma.acc, Yout, m0, rows_x, mbase, n0 + nbase, N, lane);
        } else {
            wait_lgkmcnt0();
            barrier();  // every wave is done with the ring
            epi.store_slices_lds(mma.acc, smem + wave * STAGE_BYTES, ep_xs, ep_ws, ep_b, Yout,
                                 m0, rows_x, mbase, nbase, n0, N, lane);
        }
    } else {
        EpiT epi;
        if constexpr (EPI == kStoreI32) {
            epi.store(mma.acc, Yout, m0, rows_x, mbase, n0 + nbase, N, lane & 31, lane >> 5);
        } else {
            epi.load_lds(ep_xs, ep_ws, ep_b, mbase, nbase, lane & 31, lane >> 5);
            wait_lgkmcnt0();
            barrier();  // every wave is done with the ring
            if constexpr (SLICED)
                epi.store_slices(mma.acc, smem + wave * STAGE_BYTES, Yout, m0, rows_x, mbase,
                                 n0 + nbase, N, lane & 31, lane >> 5, lane);
            else
                epi.store_rows(mma.acc, smem + wave * STAGE_BYTES, Yout, m0, rows_x, mbase,
                               n0 + nbase, N, lane & 31, lane >> 5, lane);
        }
    }
}

// --------------------------------------------------------------------------
// gemm_pt_kernel: gemm_2s_kernel's 12-wave tile (288 x 256, 96 x 64 per
// wave, four loading waves, two-slot ring of 128-byte K tiles) made
// persistent. Workgroup b walks tiles b, b + G, b + 2G, ... (G = gridDim.x,
// a multiple of 8, so every tile of a workgroup maps to the XCD it runs on
// and the tiles resident on an XCD at any time are those gemm_2s_kernel's
// round would place there). What a new workgroup would wait for is fetched
// while the previous tile drains:
//   - the next tile's first K tile is loaded at the boundary of the current
//     tile's second-to-last K tile, into the slot it frees;
//   - its second K tile right after the epilogue, into the slot that staged
//     the output rows;
//   - the epilogue operands (x_scale, w_scale, bias) by direct-to-LDS
//     dword loads from a wave that issues no tile loads, one tile ahead of
//     their use.
// Slots alternate over the workgroup's whole K-tile sequence. Each slot holds
// X then W contiguously (68 KB), so one slot can stage all 12 waves' 32-token
// output slices (55 KB). Needs 256 <= K bytes, N % 8 == 0 and w_scale / bias
// 16 / 8-byte aligned (the launcher checks).
// --------------------------------------------------------------------------
template <class Op, int EPI, bool HAS_BIAS>
__global__ __launch_bounds__(768) void gemm_pt_kernel(
    const int8_t *__restrict__ X, const int8_t *__restrict__ W, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int BM = 288, BN = 256, BK = 128, SWZ = 1, GROUP_M = 8;
    constexpr int WAVES_N = 4;
    constexpr int WTM = 96, WTN = 64;
    constexpr int TJ = WTM / 32, TI = WTN / 32;
    constexpr int NI = 4;                 // loading waves
    constexpr int EPW = NI;               // the wave that loads the epilogue operands
    constexpr int LX = BM * BK / 1024 / NI;  // 9 DMA blocks per loading wave, X
    constexpr int LW = BN * BK / 1024 / NI;  // 8, W
    constexpr int LOADS = LX + LW;
    constexpr int XSLOT = BM * BK;
    constexpr int SLOT = (BM + BN) * BK;
    constexpr int ROWS_PER_DMA = 1024 / BK;  // 8 rows of a panel per 1 KiB block
    using EpiT = Epi16<TI, TJ, EPI, true, HAS_BIAS>;
    static_assert(12 * EpiT::kSliceBytes <= SLOT, "output slices stage in one slot");
    // epilogue operands: x_scale [320] (BM rounded up to whole 64-lane
    // dword loads), w_scale [256], bias [256] bf16
    constexpr int EP_XS = 320 * 4, EP_WS = BN * 4, EP_B = BN * 2;
    constexpr int NXS = EP_XS / 256, NWS = EP_WS / 256, NB = EP_B / 256;
    static_assert(2 * SLOT + EP_XS + EP_WS + EP_B <= 160 * 1024, "LDS");

    __shared__ __attribute__((aligned(1024))) int8_t smem[2 * SLOT + EP_XS + EP_WS + EP_B];
    float *ep_xs = reinterpret_cast<float *>(smem + 2 * SLOT);
    float *ep_ws = reinterpret_cast<float *>(smem + 2 * SLOT + EP_XS);
    uint16_t *ep_b = reinterpret_cast<uint16_t *>(smem + 2 * SLOT + EP_XS + EP_WS);
    keep_args(xs, ws, bias, Yout);

    const int total = tiles_m * tiles_n;
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int mbase = (wave / WAVES_N) * WTM;
    const int nbase = (wave % WAVES_N) * WTN;
    const bool loader = wave < NI;
    const int iw = loader ? wave : 0;
    const int KT = Kb / BK;  // >= 2, the launcher guarantees BK divides Kb
    // Lane part of every DMA offset: block iw + i NI starts 32 i rows below
    // block iw, and the swizzle key of a row does not change over 32 rows.
    const uint32_t off0 = dma_offset<BK, SWZ>(iw, lane, Kb);
    const uint32_t panel_step = static_cast<uint32_t>(NI * ROWS_PER_DMA) * Kb;

    auto slot_ptr = [&](int q) { return smem + (q & 1) * SLOT; };
    struct Tile {
        int m0, n0, rows_x, rows_w;
        __amdgpu_buffer_rsrc_t rx, rw;
    };
    auto tile_of = [&](int t) {
        int tm, tn;
        map_tile<GROUP_M>(t, tiles_m, tiles_n, tm, tn);
        Tile r;
        r.m0 = tm * BM;
        r.n0 = tn * BN;
        r.rows_x = min(BM, M - r.m0);
        r.rows_w = min(BN, N - r.n0);
        r.rx = make_rsrc(X + static_cast<int64_t>(r.m0) * Kb, static_cast<uint32_t>(r.rows_x) * Kb);
        r.rw = make_rsrc(W + static_cast<int64_t>(r.n0) * Kb, static_cast<uint32_t>(r.rows_w) * Kb);
        return r;
    };
    // Load i of this wave's share of K tile kt of `tl` into the slot of
    // sequence number q: W blocks first, then X blocks.
    // (The opaque copy of off0 keeps the compiler from hoisting the 17
    // per-load sums out of the loops, which would hold 17 registers.)
    auto issue_one = [&](const Tile &tl, int kt, int q, int i) {
        if (!loader) return;
        int8_t *slot = slot_ptr(q);
        uint32_t base = off0;
        asm volatile("" : "+v"(base));
        uint32_t step = panel_step;
        asm volatile("" : "+s"(step));
        if (i < LW)
            dma16(tl.rw, slot + XSLOT + (iw + i * NI) * 1024, base + (i * step + kt * BK));
        else
            dma16(tl.rx, slot + (iw + (i - LW) * NI) * 1024, base + ((i - LW) * step + kt * BK));
    };
    // The epilogue operands of `tl` into LDS (wave EPW; zero past M / N).
    auto issue_ep = [&](const Tile &tl) {
        if (wave != EPW || EPI == kStoreI32) return;
        if constexpr (EPI == kDequantBf16) {
            const __amdgpu_buffer_rsrc_t rxs =
                make_rsrc(xs + tl.m0, static_cast<uint32_t>(tl.rows_x) * 4u);
            const __amdgpu_buffer_rsrc_t rws =
                make_rsrc(ws + tl.n0, static_cast<uint32_t>(tl.rows_w) * 4u);
#pragma unroll
            for (int i = 0; i < NXS; ++i)
                dma4(rxs, reinterpret_cast<int8_t *>(ep_xs) + 256 * i, 4u * lane + 256u * i);
#pragma unroll
            for (int i = 0; i < NWS; ++i)
                dma4(rws, reinterpret_cast<int8_t *>(ep_ws) + 256 * i, 4u * lane + 256u * i);
        }
        const __amdgpu_buffer_rsrc_t rb =
            make_rsrc(HAS_BIAS ? bias + tl.n0 : bias,
                      HAS_BIAS ? static_cast<uint32_t>(tl.rows_w) * 2u : 0u);
#pragma unroll
        for (int i = 0; i < NB; ++i)
            dma4(rb, reinterpret_cast<int8_t *>(ep_b) + 256 * i, 4u * lane + 256u * i);
    };

    Mma16<typename Narrow<Op>::type, BK, TI, TJ, SWZ> mma;
    int t = blockIdx.x;
    Tile cur = tile_of(t);
    int q = 0;  // sequence number of the current tile's first K tile

    // Prologue of the first tile: K tiles 0 and 1, its epilogue operands.
#pragma unroll
    for (int i = 0; i < LOADS; ++i) issue_one(cur, 0, 0, i);
    issue_ep(cur);
    wait_vmcnt<0>();
    barrier();
#pragma unroll
    for (int i = 0; i < LOADS; ++i) issue_one(cur, 1, 1, i);
    mma.init(lane, mbase, nbase);
    mma.template load<0>(slot_ptr(0), slot_ptr(0) + XSLOT);

    auto boundary = [&] {
        wait_lgkmcnt0();  // this wave's reads of the current slot are done
        wait_vmcnt<0>();  // and its loads of the next K tile have landed
        barrier();
    };
    for (;;) {
        const int tn_ = t + static_cast<int>(gridDim.x);
        const bool has_next = tn_ < total;
        const Tile nxt = tile_of(has_next ? tn_ : t);
        int kt = 0;
        // The boundary of K tile kt sends K tile kt+2 into the slot it frees;
        // at kt = KT-2 that is the next tile's first K tile. (One loop for
        // both keeps the register allocation of the loop body: as a separate
        // copy after the loop, the tile spilled an accumulator.)
        auto issue_ahead = [&](int i) {
            const bool same = kt + 2 < KT;
            if (same || has_next) issue_one(same ? cur : nxt, same ? kt + 2 : 0, q + kt + 2, i);
        };
        for (; kt + 1 < KT; ++kt)
            mma.template tile<false, LOADS>(slot_ptr(q + kt), slot_ptr(q + kt) + XSLOT,
                                            slot_ptr(q + kt + 1), slot_ptr(q + kt + 1) + XSLOT,
                                            boundary, issue_ahead);
        mma.template tile<true, 0>(slot_ptr(q + kt), slot_ptr(q + kt) + XSLOT,
                                   slot_ptr(q + kt), slot_ptr(q + kt) + XSLOT, [] {},
                                   [](int) {});
        // Epilogue. The slot of K tile KT-1 stages the output rows; the
        // other slot holds the next tile's first K tile.
        int8_t *stage = slot_ptr(q + KT - 1);
        wait_lgkmcnt0();
        wait_vmcnt<0>();  // loaders: the next first K tile; EPW: the operands
        barrier();
        // Lane-dependent addresses are rederived per tile from an opaque
        // copy of the lane id rather than hoisted and held across the K
        // tiles (here the epilogue's, below the next tile's fragments').
        int le = lane;
        asm volatile("" : "+v"(le));
        EpiT epi;
        if constexpr (EPI == kStoreI32) {
            epi.store(mma.acc, Yout, cur.m0, cur.rows_x, mbase, cur.n0 + nbase, N, le);
        } else {
            epi.store_slices_lds(mma.acc, stage + wave * EpiT::kSliceBytes, ep_xs, ep_ws, ep_b,
                                 Yout, cur.m0, cur.rows_x, mbase, nbase, cur.n0, N, le);
        }
        if (!has_next) break;
        wait_lgkmcnt0();
        barrier();  // staging slot and operand area free
        q += KT;
        cur = nxt;
        t = tn_;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) issue_one(cur, 1, q + 1, i);
        issue_ep(cur);
        int ln2 = lane;
        asm volatile("" : "+v"(ln2));
        mma.init(ln2, mbase, nbase);
        mma.template load<0>(slot_ptr(q), slot_ptr(q) + XSLOT);
    }
}

// --------------------------------------------------------------------------
// gemm_ws_kernel: NPROD producer waves issue the tile loads, WAVES_M x
// WAVES_N consumer waves multiply. One barrier per K tile hands slots over:
//   barrier #0: tile 0 has landed;
//   between barrier #kt and #kt+1: consumers multiply tile kt; producers
//     refill slot kt-1 (free: every consumer read of it completed before
//     barrier #kt) with tile kt+STAGES-1, then wait for tile kt+1.
// The launcher guarantees BK divides K (no K tail).
// --------------------------------------------------------------------------
template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int NPROD, int STAGES,
          int SWZ, int GROUP_M, int EPI, bool N_VEC, bool HAS_BIAS>
__global__ __launch_bounds__((WAVES_M * WAVES_N + NPROD) * 64) void gemm_ws_kernel(
    const int8_t *__restrict__ X, const int8_t *__restrict__ W, const float *__restrict__ xs,
    const float *__restrict__ ws, const uint16_t *__restrict__ bias, int M, int N, int Kb,
    void *__restrict__ Yout, int tiles_m, int tiles_n) {
    constexpr int NC = WAVES_M * WAVES_N;
    constexpr int WTM = BM / WAVES_M;
    constexpr int WTN = BN / WAVES_N;
    constexpr int TJ = WTM / 32;
    constexpr int TI = WTN / 32;
    constexpr int NBX = BM * BK / 1024;      // 1 KiB DMA blocks per stage, X tile
    constexpr int NBW = BN * BK / 1024;      // ... W tile
    constexpr int LP = (NBX + NBW) / NPROD;  // blocks per producer wave
    constexpr int STAGE = (BM + BN) * BK;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
    static_assert(LP * NPROD == NBX + NBW, "DMA split");
    static_assert(BK == 64 || BK == 128, "K tile of 64 or 128 bytes");
    static_assert(STAGES >= 2 && LP * (STAGES - 2) < 64, "vmcnt range");
    static_assert(STAGES * STAGE + 4 * BM + 6 * BN <= 160 * 1024, "LDS");

    // LDS: the ring, then the tile's epilogue operands (x_scale [BM],
    // w_scale [BN], bias [BN]).
    constexpr int EP_BYTES = 4 * BM + 4 * BN + 2 * BN;
    __shared__ __attribute__((aligned(1024))) int8_t smem[STAGES * STAGE + EP_BYTES];
    float *ep_xs = reinterpret_cast<float *>(smem + STAGES * STAGE);
    float *ep_ws = ep_xs + BM;
    uint16_t *ep_b = reinterpret_cast<uint16_t *>(ep_ws + BN);
    using EpiT = Epi<TI, TJ, EPI, N_VEC, HAS_BIAS>;
    keep_args(xs, ws, bias, Yout);

    int tm, tn;
    map_tile<GROUP_M>(blockIdx.x, tiles_m, tiles_n, tm, tn);
    const int m0 = tm * BM;
    const int n0 = tn * BN;
    const int lane = threadIdx.x & 63;
    const int wave = wave_id();
    const int rows_x = min(BM, M - m0);
    const int rows_w = min(BN, N - n0);
    const int KT = Kb / BK;

    if (wave >= NC) {
        // ---------------- producer ----------------
        const int p = wave - NC;
        const __amdgpu_buffer_rsrc_t rx =
            make_rsrc(X + static_cast<int64_t>(m0) * Kb, static_cast<uint32_t>(rows_x) * Kb);
        const __amdgpu_buffer_rsrc_t rw =
            make_rsrc(W + static_cast<int64_t>(n0) * Kb, static_cast<uint32_t>(rows_w) * Kb);
        uint32_t off[LP];
#pragma unroll
        for (int i = 0; i < LP; ++i) {
            const int b = p * LP + i;
            off[i] = dma_offset<BK, SWZ>(b < NBX ? b : b - NBX, lane, Kb);
        }
        auto issue = [&](int t) {
            int8_t *slot = smem + (t % STAGES) * STAGE;
            const int kb = t * BK;
#pragma unroll
            for (int i = 0; i < LP; ++i) {
                const int b = p * LP + i;  // X blocks first, then W blocks
                dma16(b < NBX ? rx : rw, slot + b * 1024, off[i] + kb);
            }
        };
#pragma unroll
        for (int t = 0; t < STAGES - 1; ++t)
            if (t < KT) issue(t);
        if (STAGES - 1 <= KT)
            wait_vmcnt<LP * (STAGES - 2)>();
        else
            wait_vmcnt<0>();
        barrier();  // #0
        int kt = 0;
        for (; kt + STAGES - 1 < KT; ++kt) {
            issue(kt + STAGES - 1);
            wait_vmcnt<LP * (STAGES - 2)>();  // tile kt+1 has landed
            barrier();                        // #kt+1
        }
        // Every tile load is issued: the first producer now stages the
        // epilogue operands in LDS (their latency overlaps the last tiles).
        if (EPI != kStoreI32 && p == 0) {
            EpiT::template fill_lds<BM, BN>(ep_xs, ep_ws, ep_b, xs, ws, bias, m0, rows_x, n0,
                                            rows_w, lane);
            wait_lgkmcnt0();
        }
        for (; kt + 1 < KT; ++kt) {
            wait_vmcnt<0>();
            barrier();
        }
        barrier();  // final: the epilogue operands are in LDS
        return;
    }

    // ---------------- consumer ----------------
    prefer_agpr_mfma();
    const int mbase = (wave / WAVES_N) * WTM;
    const int nbase = (wave % WAVES_N) * WTN;
    Mma<Op, BM, BK, TI, TJ, SWZ> mma;
    mma.init(lane, mbase, nbase);
    barrier();  // #0
    mma.load(smem, 0, 0);
    int kt = 0;
    for (; kt + 1 < KT; ++kt)
        mma.template tile<false>(smem + (kt % STAGES) * STAGE, [&] {
            wait_lgkmcnt0();  // every read of slot kt has completed
            barrier();        // #kt+1: tile kt+1 has landed
            mma.load(smem + ((kt + 1) % STAGES) * STAGE, 0, 0);
        });
    mma.template tile<true>(smem + (kt % STAGES) * STAGE, [] {});
    barrier();  // final: the epilogue operands are in LDS and the ring is free

    EpiT epi;
    if constexpr (EPI == kStoreI32) {
        epi.store(mma.acc, Yout, m0, rows_x, mbase, n0 + nbase, N, lane & 31, lane >> 5);
    } else {
        static_assert(NC * EpiT::kStageBytes <= STAGES * STAGE, "row staging fits the ring");
        epi.load_lds(ep_xs, ep_ws, ep_b, mbase, nbase, lane & 31, lane >> 5);
        epi.store_rows(mma.acc, smem + wave * EpiT::kStageBytes, Yout, m0, rows_x, mbase,
                       n0 + nbase, N, lane & 31, lane >> 5, lane);
    }
}

// --------------------------------------------------------------------------
// launchers
// --------------------------------------------------------------------------

struct GemmArgs {
    const int8_t *X;
    const int8_t *W;
    const float *xs;
    const float *ws;
    const uint16_t *bias;
    int M, N, Kb;
    void *Y;
    hipStream_t stream;
};

// The four instances of one configuration: vector epilogue operands (N % 4
// == 0 with aligned w_scale / bias) or not, with or without a bias.
template <template <bool, bool> class K>
hipError_t dispatch(const GemmArgs &a, int EPI_is_i32, int BM, int BN, int threads) {
    int tiles_m = (a.M + BM - 1) / BM;
    int tiles_n = (a.N + BN - 1) / BN;
    const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(tiles_m) * tiles_n));
    const bool has_bias = !EPI_is_i32 && a.bias != nullptr;
    const bool n_vec = a.N % 4 == 0 && (reinterpret_cast<uintptr_t>(a.ws) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(a.bias) & 7) == 0;
    const void *fn = n_vec ? (has_bias ? K<true, true>::fn() : K<true, false>::fn())
                           : (has_bias ? K<false, true>::fn() : K<false, false>::fn());
    const int8_t *X = a.X;
    const int8_t *W = a.W;
    const float *xs = a.xs;
    const float *ws = a.ws;
    const uint16_t *bias = a.bias;
    int M = a.M, N = a.N, Kb = a.Kb;
    void *Y = a.Y;
    void *args[] = {&X, &W, &xs, &ws, &bias, &M, &N, &Kb, &Y, &tiles_m, &tiles_n};
    return hipLaunchKernel(fn, grid, dim3(threads), args, 0, a.stream);
}

template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int STAGES, int SWZ,
          int GROUP_M, int EPI>
struct Uniform {
    template <bool NV, bool HB>
    struct K {
        static const void *fn() {
            return reinterpret_cast<const void *>(
                &gemm_kernel<Op, BM, BN, BK, WAVES_M, WAVES_N, STAGES, SWZ, GROUP_M, EPI, NV, HB>);
        }
    };
    static hipError_t launch(const GemmArgs &a) {
        if (a.Kb % BK != 0) return hipErrorInvalidValue;
        return dispatch<K>(a, EPI == kStoreI32, BM, BN, WAVES_M * WAVES_N * 64);
    }
};

template <class Op, int BM, int BN, int BK, int WAVES_M, int WAVES_N, int NPROD, int STAGES,
          int SWZ, int GROUP_M, int EPI>
struct Specialized {
    template <bool NV, bool HB>
    struct K {
        static const void *fn() {
            return reinterpret_cast<const void *>(
                &gemm_ws_kernel<Op, BM, BN, BK, WAVES_M, WAVES_N, NPROD, STAGES, SWZ, GROUP_M, EPI,
                                NV, HB>);
        }
    };
    static hipError_t launch(const GemmArgs &a) {
        if (a.Kb % BK != 0) return hipErrorInvalidValue;
        return dispatch<K>(a, EPI == kStoreI32, BM, BN, (WAVES_M * WAVES_N + NPROD) * 64);
    }
};

// The persistent 288 x 256 kernel: one workgroup per CU (a multiple of 8,
// at most one per tile), each walking its tiles.
int persistent_grid() {
    static std::atomic<int> cached[256];  // per device; racing fills agree
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 256) return 0;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        n = cus / 8 * 8;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

template <class Op, int EPI>
struct Persistent {
    template <bool HB>
    static const void *fn() {
        return reinterpret_cast<const void *>(&gemm_pt_kernel<Op, EPI, HB>);
    }
    // Whether the persistent kernel takes this launch: whole rounds of
    // 288 x 256 tiles to walk, at least two K tiles, and the vector
    // epilogue's layout (N % 8 == 0, w_scale / bias aligned).
    static bool applies(const GemmArgs &a, int grid) {
        const int64_t tiles = static_cast<int64_t>((a.M + 287) / 288) * ((a.N + 255) / 256);
        return grid >= 8 && tiles > grid && a.Kb % 128 == 0 && a.Kb >= 256 && a.N % 8 == 0 &&
               (reinterpret_cast<uintptr_t>(a.ws) & 15) == 0 &&
               (reinterpret_cast<uintptr_t>(a.bias) & 7) == 0;
    }
    static hipError_t launch(const GemmArgs &a, int grid) {
        int tiles_m = (a.M + 287) / 288;
        int tiles_n = (a.N + 255) / 256;
        const bool has_bias = EPI != kStoreI32 && a.bias != nullptr;
        const void *f = has_bias ? fn<true>() : fn<false>();
        const int8_t *X = a.X;
        const int8_t *W = a.W;
        const float *xs = a.xs;
        const float *ws = a.ws;
        const uint16_t *bias = a.bias;
        int M = a.M, N = a.N, Kb = a.Kb;
        void *Y = a.Y;
        void *args[] = {&X, &W, &xs, &ws, &bias, &M, &N, &Kb, &Y, &tiles_m, &tiles_n};
        return hipLaunchKernel(f, dim3(static_cast<unsigned>(grid)), dim3(768), args, 0,
                               a.stream);
    }
};

template <class Op, int BM, int BN, int WAVES_M, int WAVES_N, int SWZ, int GROUP_M, int EPI>
struct TwoSlot {
    template <bool NV, bool HB>
    struct K {
        static const void *fn() {
            return reinterpret_cast<const void *>(
                &gemm_2s_kernel<Op, BM, BN, WAVES_M, WAVES_N, SWZ, GROUP_M, EPI, NV, HB>);
        }
    };
    static hipError_t launch(const GemmArgs &a) {
        if (a.Kb % 128 != 0) return hipErrorInvalidValue;
        return dispatch<K>(a, EPI == kStoreI32, BM, BN, WAVES_M * WAVES_N * 64);
    }
};

// Default configurations.
//  - K a multiple of 128 bytes (every DiT shape): the candidate that
//    minimizes the estimated time, rounds of the 256 CUs (one workgroup per
//    CU) x tile area / rate, where rate is the throughput per output
//    element at full rounds, measured at 4608 x 4096 -> 16384 (where every
//    candidate fills whole rounds) relative to the 288 x 256 tiles, whose
//    16 x 16 MFMAs make them the fastest per element. Ties go to the earlier
//    candidate.
//    * 288 x 256 tiles (tokens x channels), two-slot, 12 waves of 96 x 64:
//      at M = 4608 = 16 x 288 every DiT shape fills whole rounds (N = 16384:
//      4, N = 12288: 3, N = 4096: 1);
//    * 192 x 256, two-slot, 8 waves of 96 x 64;
//    * 192 x 128 and 256 x 128, warp-specialized (4 consumer waves of 96 x
//      64 or 128 x 64, 4 producer waves, 3-slot ring): the small tiles for
//      outputs of fewer than a round of large tiles.
//    All use 128-byte K tiles (full cache lines per row) and the swizzle key
//    (row >> 1) & 7.
//  - otherwise: every wave loads, 192 x 256 tiles, 4 waves of 192 x 64,
//    4-slot ring of 64-byte K tiles (BK = 64 divides K), key (row >> 2) & 3.
struct TileChoice {
    int bm, bn, threads;
    double rate;
};
constexpr TileChoice kTiles[] = {
    {288, 256, 768, 1.0},
    {192, 256, 512, 0.82},
    {192, 128, 512, 0.71},
    {256, 128, 512, 0.73},
};
constexpr int kTileChoices = sizeof(kTiles) / sizeof(kTiles[0]);

// A candidate whose grid would reach 2^32 work-items is skipped; the first
// never does within the entry points' limit M N <= 2^38.
int pick_tiles(int M, int N) {
    int best = 0;
    double best_t = 0.0;
    for (int c = 0; c < kTileChoices; ++c) {
        const TileChoice &t = kTiles[c];
        const int64_t tiles = static_cast<int64_t>((M + t.bm - 1) / t.bm) * ((N + t.bn - 1) / t.bn);
        if (c > 0 && tiles * t.threads >= (INT64_C(1) << 32)) continue;
        const int64_t rounds = (tiles + 255) / 256;
        const double est = static_cast<double>(rounds) * t.bm * t.bn / t.rate;
        if (c == 0 || est < best_t) {
            best = c;
            best_t = est;
        }
    }
    return best;
}

template <class Op, int EPI>
hipError_t launch_default(const GemmArgs &a) {
    if (a.Kb % 128 == 0) {
        switch (pick_tiles(a.M, a.N)) {
        case 0: {
            const int grid = persistent_grid();
            if (Persistent<Op, EPI>::applies(a, grid)) return Persistent<Op, EPI>::launch(a, grid);
            return TwoSlot<Op, 288, 256, 3, 4, 1, 8, EPI>::launch(a);
        }
        case 1:
            return TwoSlot<Op, 192, 256, 2, 4, 1, 4, EPI>::launch(a);
        case 2:
            return Specialized<Op, 192, 128, 128, 2, 2, 4, 3, 1, 4, EPI>::launch(a);
        default:
            return Specialized<Op, 256, 128, 128, 2, 2, 4, 3, 1, 4, EPI>::launch(a);
        }
    }
    return Uniform<Op, 192, 256, 64, 1, 4, 4, 2, 4, EPI>::launch(a);
}

}  // namespace

hipError_t launch_gemm_i8(const int8_t *A, const int8_t *B, const float *xs, const float *ws,
                          const uint16_t *bias, int64_t M, int64_t N, int64_t K, uint16_t *Y,
                          int32_t *Y32, hipStream_t stream) {
    GemmArgs a{A, B, xs, ws, bias, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K),
               Y32 != nullptr ? static_cast<void *>(Y32) : static_cast<void *>(Y), stream};
    if (Y32 != nullptr) {
        a.xs = nullptr;
        a.ws = nullptr;
        a.bias = nullptr;
        return launch_default<I8Op, kStoreI32>(a);
    }
    return launch_default<I8Op, kDequantBf16>(a);
}

hipError_t launch_gemm_bf16(const uint16_t *A, const uint16_t *B, const uint16_t *bias,
                            int64_t M, int64_t N, int64_t K, uint16_t *Y, hipStream_t stream) {
    GemmArgs a{reinterpret_cast<const int8_t *>(A),
               reinterpret_cast<const int8_t *>(B),
               nullptr,
               nullptr,
               bias,
               static_cast<int>(M),
               static_cast<int>(N),
               static_cast<int>(2 * K),
               Y,
               stream};
    return launch_default<Bf16Op, kBiasBf16>(a);
}

void gemm_config(int64_t M, int64_t N, int64_t Kb, int *tile_m, int *tile_n, int *threads) {
    if (Kb % 128 == 0) {
        const TileChoice &t = kTiles[pick_tiles(static_cast<int>(M), static_cast<int>(N))];
        *tile_m = t.bm;
        *tile_n = t.bn;
        *threads = t.threads;
    } else {
        *tile_m = 192;
        *tile_n = 256;
        *threads = 256;
    }
}

}  // namespace w8a8
