// Device helpers shared by the convolution kernels.
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

namespace shardconv {

// bfloat16 is carried as its 16-bit pattern.
using bf16_t = uint16_t;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// binary32 -> bfloat16, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f)
{
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7f800000u) == 0x7f800000u) return bf16_t((b >> 16) | ((b & 0xffffu) ? 0x40u : 0u));
    b += 0x7fffu + ((b >> 16) & 1u);
    return bf16_t(b >> 16);
}

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// Workgroups are dispatched round-robin over the 8 XCDs of an MI355X, each
// with its own L2. Remap the dispatch index so that XCD x runs a contiguous
// range of logical block indices (neighbouring tiles share halo rows in L2).
// Bijective on [0, nblocks) for any nblocks.
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nblocks)
{
    constexpr int64_t kXcd = 8;
    const int64_t x = b % kXcd, j = b / kXcd;
    const int64_t q = nblocks / kXcd, r = nblocks % kXcd;
    return x * q + (x < r ? x : r) + j;
}

}  // namespace shardconv
