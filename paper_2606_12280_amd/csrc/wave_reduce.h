// Reductions over the 64 lanes of a wave that leave the result in every
// lane, through DPP lane exchanges instead of LDS permutes: quad_perm
// [1,0,3,2] and [2,3,0,1] (lanes xor 1 and xor 2), row_half_mirror (lane i
// <-> 7-i within each 8) and row_mirror (i <-> 15-i within each 16) leave
// every lane of a 16-lane row with the row's total; the four rows are then
// combined in one fixed order from lanes 0, 16, 32 and 48, so every lane
// holds the same bits. Each exchange is a VALU operation of a few cycles'
// latency, against about a hundred for a ds_bpermute round trip.
//
// All four patterns are permutations inside a row, so every lane reads a
// valid source lane and the DPP "old" operand is never used: the exchanges
// are issued with it undefined and bound_ctrl set, which spares the
// register the compiler would otherwise zero before each exchange.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {
namespace lanes {

constexpr int kXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141; // row_half_mirror
constexpr int kMirror = 0x140;     // row_mirror

template <int CTRL>
__device__ __forceinline__ unsigned dpp_u32(unsigned v) {
    return static_cast<unsigned>(
        __builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xF, 0xF, true));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long b = __double_as_longlong(v);
    const unsigned lo = dpp_u32<CTRL>(static_cast<unsigned>(b));
    const unsigned hi = dpp_u32<CTRL>(static_cast<unsigned>(b >> 32));
    return __longlong_as_double((static_cast<long long>(hi) << 32) | lo);
}

__device__ __forceinline__ unsigned lane_u32(unsigned v, int l) {
    return static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(v), l));
}

__device__ __forceinline__ double lane_f64(double v, int l) {
    const long long b = __double_as_longlong(v);
    const unsigned lo = lane_u32(static_cast<unsigned>(b), l);
    const unsigned hi = lane_u32(static_cast<unsigned>(b >> 32), l);
    return __longlong_as_double((static_cast<long long>(hi) << 32) | lo);
}

// Maximum of an absmax: v must lie in [+0, +inf] (never negative, never
// NaN), as a running fmaxf of fabsf values started from 0 does. On that
// range the IEEE-754 order equals the unsigned order of the bit patterns,
// so the maximum is taken as an integer maximum, which folds each exchange
// into a single v_max_u32 with DPP (a float maximum would also canonicalize
// both operands first) and gives exactly what fmaxf gives.
__device__ __forceinline__ float max_nonneg(float f) {
    unsigned v = __float_as_uint(f);
    v = ::max(v, dpp_u32<kXor1>(v));
    v = ::max(v, dpp_u32<kXor2>(v));
    v = ::max(v, dpp_u32<kHalfMirror>(v));
    v = ::max(v, dpp_u32<kMirror>(v));
    const unsigned a = ::max(lane_u32(v, 0), lane_u32(v, 16));
    const unsigned b = ::max(lane_u32(v, 32), lane_u32(v, 48));
    return __uint_as_float(::max(a, b));
}

__device__ __forceinline__ double sum(double v) {
    v += dpp_f64<kXor1>(v);
    v += dpp_f64<kXor2>(v);
    v += dpp_f64<kHalfMirror>(v);
    v += dpp_f64<kMirror>(v);
    return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}

}  // namespace lanes
}  // namespace w8a8
