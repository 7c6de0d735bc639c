// Memory access and code packing shared by the row kernels (the W8A8
// activation quantization and its adaLN-fused form).
//
// Row loads and stores go through raw buffer instructions with a per-row
// resource: a lane whose chunk lies past the row, or a row past the input,
// falls outside the resource's range, so the hardware reads zeros and drops
// the store. Every wave then issues the same memory instructions for every
// row, with no branch around them. That matters: around a conditional load
// the compiler cannot count the loads in flight and waits for all of them,
// which made a prefetched next row arrive before the current one was used.
// With straight-line memory instructions it waits for the current row only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace w8a8 {
namespace rows {

constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format
constexpr int kNontemporal = 2;           // nt: streamed, not kept in the caches

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, static_cast<int>(bytes),
                                             kBufferWord3);
}

// 16 bytes at byte offset off (zeros when out of range).
__device__ __forceinline__ uint4 load_chunk(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNontemporal);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// 8 codes at byte offset off (dropped when out of range).
__device__ __forceinline__ void store_codes(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t lo,
                                            uint32_t hi) {
    const v2u v = {lo, hi};
    __builtin_amdgcn_raw_buffer_store_b64(v, r, off, 0, kNontemporal);
}

__device__ __forceinline__ void store_f32(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, 0);
}

// The wave's index in its workgroup, in a scalar register: values derived
// from it (row indices, buffer resources) are then wave-uniform to the
// compiler, which otherwise loops over the lanes to build a resource.
__device__ __forceinline__ int wave_index() {
    return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
}

// The code of v at multiplier r, clamp(rint(v * r), -127, 127), in the low
// byte of the returned word: the product is clamped first (rint is monotone
// and the bounds are integers, so the order does not matter; a NaN product
// clamps to -127 either way), then adding 1.5 * 2^23 rounds it to the nearest
// integer, ties to even, and leaves that integer in two's complement in the
// low mantissa bits.
__device__ __forceinline__ uint32_t code_word(float v, float r) {
    const float c = fminf(fmaxf(v * r, -127.0f), 127.0f);
    return __float_as_uint(c + 0x1.8p23f);
}

// The low bytes of four words, a in byte 0 (three v_perm_b32).
__device__ __forceinline__ uint32_t pack4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    const uint32_t ab = __builtin_amdgcn_perm(b, a, 0x0c0c0400u);
    const uint32_t cd = __builtin_amdgcn_perm(d, c, 0x0c0c0400u);
    return __builtin_amdgcn_perm(cd, ab, 0x05040100u);
}

// Row groups the current device holds at once for `kernel` launched with
// `threads` per workgroup and `groups_per_block` groups in each (CUs x
// resident workgroups per CU x groups per workgroup); 0 when the runtime
// cannot say. `cache` is the caller's, one entry per device; host threads
// calling at once may both fill an entry, with the same value.
inline int64_t resident_groups(const void *kernel, int threads, int groups_per_block,
                               std::atomic<int64_t> (&cache)[256]) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 256) return 0;
    int64_t n = cache[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        int cus = 0;
        int per_cu = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) !=
                hipSuccess)
            return 0;
        n = static_cast<int64_t>(cus) * per_cu * groups_per_block;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Rows per group for R rows: one round of the resident groups, each walking
// an equal share (at least one row).
inline int64_t rows_per_group(int64_t R, int64_t resident) {
    if (resident <= 0) resident = 256;
    return (R + resident - 1) / resident;
}

}  // namespace rows
}  // namespace w8a8
