// Halo pack / unpack / zero-fill: a box copy between a padded tile and a dense
// slab (the two halves of the halo exchange a shard performs before its local
// convolution, ShardTensor section "PyTorch Dispatch").
//
// The box is `rows` runs of `run` contiguous bytes (contiguous inner axes are
// merged on the host), seen as a sequence of V-byte vectors cut into chunks of
// kThreads * U vectors (64 KiB for 16-byte vectors). A workgroup moves whole
// chunks, each thread U vectors of it, all loads issued before any store;
// consecutive lanes touch consecutive vectors, so every wave instruction covers
// 64*V contiguous bytes and a workgroup's accesses stay within one chunk (this
// measured faster than spreading a thread's vectors over the whole box).
// Stores are nontemporal (a slab or margin is written once per exchange and
// not read again by this kernel) and loads are ordinary cached loads: on cold
// data (8 rotating buffer sets of a 2 x 16 MiB pair) ordinary loads with
// nontemporal stores moved the pair in 10.9-11.1 us, nontemporal loads and
// stores in 12.6 us, ordinary loads and stores in 13.4 us. A single-run box (the common case of a slab along the outermost
// sharded axis, which is one contiguous block of the tile) takes a
// specialisation with no index arithmetic.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {
namespace {

struct CopyArgs {
    const char* src;
    char* dst;
    int64_t base;        // tile byte offset of the first run
    int64_t cnt1, cnt2;  // inner two outer counts (cnt0 is implied by total)
    int64_t t0, t1, t2;  // tile byte strides of the three outer dims
    int64_t nvec_row;    // vectors per run
    int64_t total;       // total vectors
    int dir;             // CopyDir
};

constexpr int kThreads = 512;

template <int V>
struct Vec;
template <>
struct Vec<16> {
    using T = __attribute__((ext_vector_type(4))) unsigned int;
    static constexpr int U = 8;
};
template <>
struct Vec<4> {
    using T = uint32_t;
    static constexpr int U = 4;
};
template <>
struct Vec<2> {
    using T = uint16_t;
    static constexpr int U = 4;
};

template <int V, bool kSingleRun>
__device__ __forceinline__ int64_t tile_offset(const CopyArgs& a, int64_t v)
{
    if (kSingleRun) return a.base + v * V;
    const int64_t row = v / a.nvec_row;
    const int64_t col = v - row * a.nvec_row;
    const int64_t i2 = row % a.cnt2;
    const int64_t r1 = row / a.cnt2;
    const int64_t i1 = r1 % a.cnt1;
    const int64_t i0 = r1 / a.cnt1;
    return a.base + i0 * a.t0 + i1 * a.t1 + i2 * a.t2 + col * V;
}

// One launch copies one or two boxes (both faces of an axis): blocks below
// nblk0 take box 0, the rest box 1. The fields of a block's box are picked by
// scalar selects (a dynamic index into the kernel arguments would copy them to
// private memory).
struct CopyArgs2 {
    CopyArgs b0, b1;
    int64_t nblk0;
};

__device__ __forceinline__ CopyArgs pick_box(const CopyArgs2& aa, bool second)
{
    CopyArgs a;
    a.src = second ? aa.b1.src : aa.b0.src;
    a.dst = second ? aa.b1.dst : aa.b0.dst;
    a.base = second ? aa.b1.base : aa.b0.base;
    a.cnt1 = second ? aa.b1.cnt1 : aa.b0.cnt1;
    a.cnt2 = second ? aa.b1.cnt2 : aa.b0.cnt2;
    a.t0 = second ? aa.b1.t0 : aa.b0.t0;
    a.t1 = second ? aa.b1.t1 : aa.b0.t1;
    a.t2 = second ? aa.b1.t2 : aa.b0.t2;
    a.nvec_row = second ? aa.b1.nvec_row : aa.b0.nvec_row;
    a.total = second ? aa.b1.total : aa.b0.total;
    a.dir = second ? aa.b1.dir : aa.b0.dir;
    return a;
}

template <int V, bool kSingleRun>
__global__ __launch_bounds__(kThreads) void box_copy_kernel(CopyArgs2 aa)
{
    using T = typename Vec<V>::T;
    constexpr int kUnroll = Vec<V>::U;
    const bool second = int64_t(blockIdx.x) >= aa.nblk0;
    const CopyArgs a = pick_box(aa, second);
    const int64_t nblk = second ? int64_t(gridDim.x) - aa.nblk0 : aa.nblk0;
    const int64_t blk = second ? int64_t(blockIdx.x) - aa.nblk0 : int64_t(blockIdx.x);
    constexpr int64_t kChunk = int64_t(kThreads) * kUnroll;
    for (int64_t v0 = blk * kChunk + threadIdx.x; v0 < a.total; v0 += nblk * kChunk) {
        T val[kUnroll];
        int64_t off[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + u * kThreads;
            off[u] = v < a.total ? tile_offset<V, kSingleRun>(a, v) : 0;
            if (v < a.total) {
                if (a.dir == TILE_TO_SLAB) {
                    val[u] = *reinterpret_cast<const T*>(a.src + off[u]);
                } else if (a.dir == SLAB_TO_TILE) {
                    val[u] = *reinterpret_cast<const T*>(a.src + v * V);
                } else {
                    val[u] = T{};
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + u * kThreads;
            if (v < a.total) {
                if (a.dir == TILE_TO_SLAB) {
                    __builtin_nontemporal_store(val[u], reinterpret_cast<T*>(a.dst + v * V));
                } else {
                    __builtin_nontemporal_store(val[u], reinterpret_cast<T*>(a.dst + off[u]));
                }
            }
        }
    }
}

template <int V>
CopyArgs copy_args_v(const BoxCopy& b, CopyDir dir, const void* src, void* dst)
{
    CopyArgs a;
    a.src = static_cast<const char*>(src);
    a.dst = static_cast<char*>(dst);
    a.base = b.base;
    a.cnt1 = b.cnt[1];
    a.cnt2 = b.cnt[2];
    a.t0 = b.tstride[0];
    a.t1 = b.tstride[1];
    a.t2 = b.tstride[2];
    a.nvec_row = b.run / V;
    a.total = b.cnt[0] * b.cnt[1] * b.cnt[2] * a.nvec_row;
    a.dir = dir;
    return a;
}

template <int V>
int64_t copy_blocks(const CopyArgs& a)
{
    const int64_t per_block = int64_t(kThreads) * Vec<V>::U;
    return std::max<int64_t>(1, std::min<int64_t>(ceil_div(a.total, per_block), 1 << 20));
}

// boxes n (1 or 2) in one launch
template <int V>
hipError_t launch_v(const BoxCopy* const* b, const CopyDir* dir, const void* const* src, void* const* dst, int n,
                    hipStream_t s)
{
    CopyArgs2 aa{};
    aa.b0 = copy_args_v<V>(*b[0], dir[0], src[0], dst[0]);
    aa.b1 = n > 1 ? copy_args_v<V>(*b[1], dir[1], src[1], dst[1]) : aa.b0;
    aa.nblk0 = copy_blocks<V>(aa.b0);
    const int64_t blocks = aa.nblk0 + (n > 1 ? copy_blocks<V>(aa.b1) : 0);
    bool single = true;
    for (int i = 0; i < n; ++i) single = single && b[i]->cnt[0] * b[i]->cnt[1] * b[i]->cnt[2] == 1;
    void* args[] = {&aa};
    const void* fn = single ? reinterpret_cast<const void*>(&box_copy_kernel<V, true>)
                            : reinterpret_cast<const void*>(&box_copy_kernel<V, false>);
    return hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(kThreads), args, 0, s);
}

// tile[box] += slab, element-wise in binary32 (bf16 sums rounded to nearest
// even): the receiving half of the reverse halo exchange. One launch adds one
// or two boxes (both faces of an axis; they never overlap in one launch), split
// over the blocks like box_copy_kernel.
template <int V, typename E, bool kSingleRun>
__global__ __launch_bounds__(kThreads) void box_add_kernel(CopyArgs2 aa)
{
    using T = typename Vec<V>::T;
    constexpr int kUnroll = Vec<V>::U;
    constexpr int NE = V / int(sizeof(E));
    const bool second = int64_t(blockIdx.x) >= aa.nblk0;
    const CopyArgs a = pick_box(aa, second);
    const int64_t nblk = second ? int64_t(gridDim.x) - aa.nblk0 : aa.nblk0;
    const int64_t blk = second ? int64_t(blockIdx.x) - aa.nblk0 : int64_t(blockIdx.x);
    constexpr int64_t kChunk = int64_t(kThreads) * kUnroll;
    for (int64_t v0 = blk * kChunk + threadIdx.x; v0 < a.total; v0 += nblk * kChunk) {
        T sv[kUnroll], tv[kUnroll];
        int64_t off[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + u * kThreads;
            off[u] = v < a.total ? tile_offset<V, kSingleRun>(a, v) : 0;
            if (v < a.total) {
                sv[u] = *reinterpret_cast<const T*>(a.src + v * V);
                tv[u] = *reinterpret_cast<const T*>(a.dst + off[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t v = v0 + u * kThreads;
            if (v < a.total) {
                E es[NE], et[NE];
                __builtin_memcpy(es, &sv[u], V);
                __builtin_memcpy(et, &tv[u], V);
#pragma unroll
                for (int i = 0; i < NE; ++i) et[i] = from_f32<E>(to_f32(et[i]) + to_f32(es[i]));
                T r;
                __builtin_memcpy(&r, et, V);
                __builtin_nontemporal_store(r, reinterpret_cast<T*>(a.dst + off[u]));
            }
        }
    }
}

template <int V, typename E>
hipError_t launch_add_v(const BoxCopy* const* b, const void* const* slab, void* tile, int n, hipStream_t s)
{
    CopyArgs2 aa{};
    aa.b0 = copy_args_v<V>(*b[0], SLAB_TO_TILE, slab[0], tile);
    aa.b1 = n > 1 ? copy_args_v<V>(*b[1], SLAB_TO_TILE, slab[1], tile) : aa.b0;
    aa.nblk0 = copy_blocks<V>(aa.b0);
    const int64_t blocks = aa.nblk0 + (n > 1 ? copy_blocks<V>(aa.b1) : 0);
    bool single = true;
    for (int i = 0; i < n; ++i) single = single && b[i]->cnt[0] * b[i]->cnt[1] * b[i]->cnt[2] == 1;
    void* args[] = {&aa};
    const void* fn = single ? reinterpret_cast<const void*>(&box_add_kernel<V, E, true>)
                            : reinterpret_cast<const void*>(&box_add_kernel<V, E, false>);
    return hipLaunchKernel(fn, dim3(unsigned(blocks)), dim3(kThreads), args, 0, s);
}

}  // namespace

hipError_t launch_box_adds(const BoxCopy* const* b, int esz, const void* const* slab, void* tile, int n,
                           hipStream_t s)
{
    // the widest vector every box, the tile and the slabs allow
    auto ok = [&](int64_t v) {
        if ((reinterpret_cast<uintptr_t>(tile) % v) != 0) return false;
        for (int i = 0; i < n; ++i) {
            const BoxCopy& x = *b[i];
            if ((x.base % v) != 0 || (x.run % v) != 0 || (x.tstride[0] % v) != 0 || (x.tstride[1] % v) != 0 ||
                (x.tstride[2] % v) != 0 || (reinterpret_cast<uintptr_t>(slab[i]) % v) != 0)
                return false;
        }
        return true;
    };
    if (esz == 2) {
        if (ok(16)) return launch_add_v<16, bf16_t>(b, slab, tile, n, s);
        if (ok(4)) return launch_add_v<4, bf16_t>(b, slab, tile, n, s);
        return launch_add_v<2, bf16_t>(b, slab, tile, n, s);
    }
    if (ok(16)) return launch_add_v<16, float>(b, slab, tile, n, s);
    return launch_add_v<4, float>(b, slab, tile, n, s);
}

hipError_t launch_box_add(const BoxCopy& b, int esz, const void* slab, void* tile, hipStream_t s)
{
    const BoxCopy* bp = &b;
    return launch_box_adds(&bp, esz, &slab, tile, 1, s);
}

hipError_t launch_box_copies(const BoxCopy* const* b, const CopyDir* dir, const void* const* src, void* const* dst,
                             int n, hipStream_t s)
{
    // the widest vector every box, tile and slab of the launch allows
    auto ok = [&](int64_t v) {
        for (int i = 0; i < n; ++i) {
            const uintptr_t tile_ptr = reinterpret_cast<uintptr_t>(dir[i] == TILE_TO_SLAB ? src[i] : dst[i]);
            const uintptr_t slab_ptr = reinterpret_cast<uintptr_t>(dir[i] == TILE_TO_SLAB ? dst[i] : src[i]);
            const BoxCopy& x = *b[i];
            if ((x.base % v) != 0 || (x.run % v) != 0 || (x.tstride[0] % v) != 0 || (x.tstride[1] % v) != 0 ||
                (x.tstride[2] % v) != 0 || (tile_ptr % v) != 0 || (dir[i] != ZERO_TILE && (slab_ptr % v) != 0))
                return false;
        }
        return true;
    };
    if (ok(16)) return launch_v<16>(b, dir, src, dst, n, s);
    if (ok(4)) return launch_v<4>(b, dir, src, dst, n, s);
    return launch_v<2>(b, dir, src, dst, n, s);
}

hipError_t launch_box_copy(const BoxCopy& b, CopyDir dir, const void* src, void* dst, hipStream_t s)
{
    const BoxCopy* bp = &b;
    return launch_box_copies(&bp, &dir, &src, &dst, 1, s);
}

}  // namespace shardconv
