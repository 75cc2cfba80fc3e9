// Device helpers shared by the convolution kernels.
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

namespace shardconv {

// bfloat16 is carried as its 16-bit pattern.
using bf16_t = uint16_t;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// binary32 -> bfloat16, round to nearest even (NaN stays a NaN): the hardware
// conversion (v_cvt_pk_bf16_f32), one instruction instead of the integer
// rounding sequence.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, __bf16(f)); }

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

// Brick raster of the persistent W-march kernels. Brick t (W segment already
// removed) of a batch item's NBZ x NBY brick grid lies in raster block t / (TZ*TY)
// (blocks row-major over the grid, each TZ x TY bricks, TZ | NBZ and TY | NBY) at
// row-major position t % (TZ*TY) inside it. A workgroup handles bricks L, L + G,
// ...; with xcd_remap the 32 workgroups of an XCD hold 32 consecutive bricks, so
// a 32-brick block keeps the halo rows its bricks share in that XCD's L2, and the
// eight XCDs work on adjacent blocks at the same time (shared halos meet in the
// last-level cache). TZ = TY = 1 is the plain row-major order.
__device__ __forceinline__ void brick_rows(uint32_t t, int32_t NBZ, int32_t NBY, int32_t TZ, int32_t TY, int32_t& bz,
                                           int32_t& by, uint32_t& nn)
{
    const uint32_t per_item = uint32_t(NBZ) * uint32_t(NBY);
    nn = t / per_item;
    const uint32_t tt = t - nn * per_item;
    const uint32_t bs = uint32_t(TZ) * uint32_t(TY);
    const uint32_t blk = tt / bs, r = tt - blk * bs;
    const uint32_t nty = uint32_t(NBY) / uint32_t(TY);
    const uint32_t bzb = blk / nty, byb = blk - bzb * nty;
    const uint32_t rz = r / uint32_t(TY);
    bz = int32_t(bzb * uint32_t(TZ) + rz);
    by = int32_t(byb * uint32_t(TY) + (r - rz * uint32_t(TY)));
}

// Largest raster block TZ x TY of at most `want_z` x (32 / TZ) bricks that
// divides the NBZ x NBY grid (powers of two).
inline void pick_raster(int64_t NBZ, int64_t NBY, int want_z, int32_t& TZ, int32_t& TY)
{
    TZ = 1;
    while (TZ * 2 <= want_z && NBZ % (TZ * 2) == 0) TZ *= 2;
    TY = 1;
    while (TZ * TY * 2 <= 32 && NBY % (TY * 2) == 0) TY *= 2;
}

// W segments of the persistent W-march kernels. `rows` brick rows of `ntiles`
// tiles each are cut into segments of T tiles that `cus` workgroups take in
// rounds; a segment after a row's first pays `warm` extra tiles (the forward
// kernel rebuilds its carry). Picks the segment count with the fewest tile-steps
// per workgroup, ceil(rows * nseg / cus) * (T + warm), preferring fewer segments,
// and segments of at least `min_t` tiles. Returns nseg (the segments actually
// formed, ceil(ntiles / T)) and T.
inline void pick_segments(int64_t rows, int64_t ntiles, int64_t cus, int64_t warm, int64_t min_t, int64_t& nseg,
                          int64_t& T)
{
    nseg = 1;
    T = ntiles;
    int64_t best = ((rows + cus - 1) / cus) * ntiles;
    for (int64_t k = 2; k <= 64; ++k) {
        const int64_t t = (ntiles + k - 1) / k;
        if (t < min_t) break;
        const int64_t segs = (ntiles + t - 1) / t;
        const int64_t cost = ((rows * segs + cus - 1) / cus) * (t + warm);
        if (cost < best) {
            best = cost;
            nseg = segs;
            T = t;
        }
    }
}

}  // namespace shardconv

namespace shardconv {

// Wait until at most N vector-memory operations of this wave are outstanding
// and all its LDS operations are done, then barrier. Unlike __syncthreads(),
// this does not wait for the wave's outstanding global stores (N of them may
// still be in flight) - those need no ordering with the LDS data the barrier
// publishes (direct global->LDS loads complete in issue order before them).
template <int N>
__device__ __forceinline__ void wait_vm_barrier()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// LDS accesses issued through inline asm. The compiler's wait insertion cannot
// tell the buffers of direct global->LDS loads apart, so it would place an
// s_waitcnt vmcnt(0) before any LDS access it sees after such a load - waiting
// for every prefetch in flight. Accesses written as asm are invisible to it; the
// caller orders them itself: lds_wait<N>() waits until at most N LDS operations
// of the wave are outstanding (LDS operations complete in issue order), and
// lds_ready() marks a register as produced at that point so that no use of it
// is scheduled earlier.
typedef __attribute__((ext_vector_type(4))) unsigned int lds_u32x4;

__device__ __forceinline__ uint32_t lds_addr(const void* p)
{
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) char*)(p)));
}

template <int OFF = 0>
__device__ __forceinline__ lds_u32x4 lds_read_b128(uint32_t addr)
{
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    lds_u32x4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
    return r;
}

// ds_read_b64_tr_b16: within each 16-lane group, lane i addresses row i / 4,
// columns 4 * (i % 4) .. + 3 of a row-major 16-bit matrix, and lane j receives
// column j of the four rows.
template <int OFF = 0>
__device__ __forceinline__ uint2 lds_read_tr16_b64(uint32_t addr)
{
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    uint2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
    return r;
}

template <int OFF = 0>
__device__ __forceinline__ void lds_write_b16(uint32_t addr, uint32_t v)
{
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    asm volatile("ds_write_b16 %0, %1 offset:%2" ::"v"(addr), "v"(v), "n"(OFF) : "memory");
}

template <int OFF = 0>
__device__ __forceinline__ void lds_write_b16_hi(uint32_t addr, uint32_t v)
{
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    asm volatile("ds_write_b16_d16_hi %0, %1 offset:%2" ::"v"(addr), "v"(v), "n"(OFF) : "memory");
}

template <int N>
__device__ __forceinline__ void lds_wait()
{
    static_assert(N >= 0 && N < 16, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}

template <typename T>
__device__ __forceinline__ void lds_ready(T& v)
{
    asm volatile("" : "+v"(v));
}

// A 32-bit LDS word read now (waits for it and every earlier LDS operation of
// the wave), made wave-uniform: for polling counters that other waves raise.
__device__ __forceinline__ uint32_t lds_read_u32_now(uint32_t addr)
{
    uint32_t v;
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr) : "memory");
    return __builtin_amdgcn_readfirstlane(v);
}

// Atomic add to a 32-bit LDS word (no return value); callers issue it from one lane.
__device__ __forceinline__ void lds_add_u32(uint32_t addr, uint32_t v)
{
    asm volatile("ds_add_u32 %0, %1" ::"v"(addr), "v"(v) : "memory");
}

}  // namespace shardconv
