// Reductions over the 64 lanes of a wave that leave the result in every
// lane, through DPP lane exchanges instead of LDS permutes: quad_perm
// [1,0,3,2] and [2,3,0,1] (lanes xor 1 and xor 2), row_half_mirror (lane i
// <-> 7-i within each 8) and row_mirror (i <-> 15-i within each 16) leave
// every lane of a 16-lane row with the row's total; the four rows are then
// combined in one fixed order from lanes 0, 16, 32 and 48, so every lane
// holds the same bits. Each exchange is a VALU operation of a few cycles'
// latency, against about a hundred for a ds_bpermute round trip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {
namespace lanes {

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(
        __builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(b), CTRL, 0xF, 0xF, false);
    const int hi =
        __builtin_amdgcn_update_dpp(0, static_cast<int>(b >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((static_cast<long long>(hi) << 32) |
                                static_cast<unsigned int>(lo));
}

__device__ __forceinline__ float lane_f32(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

__device__ __forceinline__ double lane_f64(double v, int l) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane(static_cast<int>(b), l);
    const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), l);
    return __longlong_as_double((static_cast<long long>(hi) << 32) |
                                static_cast<unsigned int>(lo));
}

constexpr int kXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141; // row_half_mirror
constexpr int kMirror = 0x140;     // row_mirror

__device__ __forceinline__ float max(float v) {
    v = fmaxf(v, dpp_f32<kXor1>(v));
    v = fmaxf(v, dpp_f32<kXor2>(v));
    v = fmaxf(v, dpp_f32<kHalfMirror>(v));
    v = fmaxf(v, dpp_f32<kMirror>(v));
    return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
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
