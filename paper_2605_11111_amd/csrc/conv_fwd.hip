// Forward convolution over a padded tile as an implicit GEMM on MFMA.
//
// GEMM view: M = output voxels, N = output channels, K = taps x input
// channels. Nothing is materialised: a workgroup owns an output brick of
// BO0 x BO1 x BO2 voxels (flattened row-major, W fastest) and all-or-part of
// the output channels. It stages the brick's input footprint (the brick grown
// by the kernel reach, which is where the halo margins of the tile enter) in
// LDS once per channel pass, then every tap reads its A operand from that LDS
// copy at a shifted voxel offset; out-of-tile voxels are written as zeros while
// staging, which is the zero padding on unsharded axes.
//
// MFMA operand layout (32x32 output tile, 64 lanes, lane group g = lane/32):
//   bf16 v_mfma_f32_32x32x16_bf16: lane holds 8 consecutive K (= 8 channels of
//        one voxel) for row lane%32 -> one 16-byte LDS read per lane.
//   f32  v_mfma_f32_32x32x2_f32: lane holds 1 K value; four MFMAs consume one
//        16-byte read of 4 consecutive channels (K order permuted so that lane
//        group g of step s holds channel 8*c + 4*g + s in both operands).
// The B operand (weights) is pre-arranged by `wfrag_kernel` so that one
// coalesced 1 KiB load per wave yields a ready fragment.
//
// LDS layout: voxel v of the input brick occupies NQ 16-byte units, stored
// unit-major: unit q of voxel v at q * NV + v (NV the brick's voxels), so that
// lanes reading consecutive voxels read consecutive 16-byte words and a lane's
// address for a tap is its own fixed part plus a uniform offset.
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

struct FwdArgs {
    const char* tile;
    const uint4* wfrag;
    char* y;
    int64_t n, cin, cout;
    int64_t P[3];      // padded tile extents
    int64_t O[3];      // output extents
    int32_t K[3], S[3], pad[3];
    int32_t BO[3];     // output brick
    int32_t BI[3];     // input brick
    int32_t NB[3];     // bricks per axis
    int32_t nq;        // 16-byte units per voxel in LDS (per pass)
    int32_t cc;        // channels per pass
    int32_t npass;
    int32_t nkc;       // K-chunks over all input channels
    int32_t nt;        // 32-wide N tiles over all output channels
    int32_t ng;        // N groups (workgroups along N)
    int32_t vec;       // 16-byte loads allowed (tile base and channel rows aligned)
    int32_t yvec;      // 16-byte output stores allowed (y, the output map and cout aligned)
    int32_t rperm;     // M-tile rows take voxels transposed (see rows_transposed; needs yvec)
    int64_t nblocks;
    int64_t ybase, ys[4];  // output map: element of (n, o0, o1, o2, co) = ybase + n*ys0 + ... + co
    int64_t org[3];        // origin of the computed region of outputs (O is its extent)
    Fold fold;             // halo folded into the loads when fold.mask != 0
};

// One launch over two to four output regions of the same plan family (the
// boundary slabs of a split forward): blocks [0, end[0]) take region 0, blocks
// [end[0], end[1]) region 1, and so on (the ends of absent regions repeat the
// total).
constexpr int kMaxRegions = 4;
struct FwdLaunch {
    FwdArgs r[kMaxRegions];
    int64_t end[kMaxRegions - 1];
};

struct PlanF {
    int rm, rn;
    FwdArgs a;
    size_t lds;
    bool ok;
};

template <typename T>
struct Traits;
template <>
struct Traits<bf16_t> {
    static constexpr int kc = 16;  // channels per MFMA K-chunk
    static constexpr int esz = 2;
};
template <>
struct Traits<float> {
    static constexpr int kc = 8;
    static constexpr int esz = 4;
};

// Stage every 16-byte unit (voxel v = (z, y, x) of the brick, channel unit q)
// once across the block: fetch(v, q, z, y, x) gives its value, stored at
// lds[q * nvp + v]. A thread fetches kStageBatch units before it stores them,
// so that their loads are in flight together (one at a time, each store
// waited for its load). When a (z, y) row of units fits the block, a thread
// keeps its column (x, q) and steps over rows: one division per row instead of
// three per unit.
constexpr int kStageBatch = 4;

template <typename F>
__device__ __forceinline__ void stage_units(const FwdArgs& a, uint4* lds, int nvp, F&& fetch)
{
    constexpr int B = kStageBatch;
    const int nq = a.nq;
    const int rowlen = a.BI[2] * nq;
    if (rowlen <= kThreads) {
        const int rpp = kThreads / rowlen;
        const int r0 = int(threadIdx.x) / rowlen, cu = int(threadIdx.x) - r0 * rowlen;
        if (r0 >= rpp) return;
        const int x = cu / nq, q = cu - x * nq;
        const int rows = a.BI[0] * a.BI[1];
        for (int r = r0; r < rows; r += B * rpp) {
            uint4 val[B];
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int rr = r + j * rpp;
                val[j] = make_uint4(0, 0, 0, 0);
                if (rr < rows) {
                    const int z = rr / a.BI[1], y = rr - z * a.BI[1];
                    val[j] = fetch(rr * a.BI[2] + x, q, z, y, x);
                }
            }
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int rr = r + j * rpp;
                if (rr < rows) lds[q * nvp + rr * a.BI[2] + x] = val[j];
            }
        }
        return;
    }
    const int total = a.BI[0] * a.BI[1] * a.BI[2] * nq;
    for (int u = threadIdx.x; u < total; u += B * kThreads) {
        uint4 val[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int uu = u + j * kThreads;
            val[j] = make_uint4(0, 0, 0, 0);
            if (uu < total) {
                const int q = uu % nq, v = uu / nq;
                const int x = v % a.BI[2], yz = v / a.BI[2];
                val[j] = fetch(v, q, yz / a.BI[1], yz % a.BI[1], x);
            }
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int uu = u + j * kThreads;
            if (uu < total) lds[(uu % nq) * nvp + uu / nq] = val[j];
        }
    }
}

// Row-mode staging of a brick, when a (z, y) row of 16-byte units fits the
// block and every unit is a whole aligned vector: a thread keeps its column
// (x, q) and steps over rows, with (z, y), its place in LDS and (where the
// source buffer cannot change from row to row) the row's byte offset
// advanced by increments and the bounds tested in 32 bits: no division and,
// on the plain path, no 64-bit product per unit. The same units as
// stage_units' row mode, in the same places. FK < 0: the tile alone (a brick
// that reaches no folded margin); FK = k: margins folded on axis k only, a
// voxel coming from the tile or from the slab of its side (the tile's layout
// with axis k cut to the margin). Along W (k = 2) the column decides the
// buffer; along D or H the row does, and its offset is formed per unit.
template <typename T, int B, int FK>
__device__ __forceinline__ void stage_rows(const FwdArgs& a, uint4* lds, int nvp, int64_t nn, const int64_t i0[3],
                                           int c0)
{
    constexpr int kPerUnit = 16 / Traits<T>::esz;
    constexpr int64_t esz = Traits<T>::esz;
    // the thread's column is formed anew in every pass (an opaque copy of the
    // thread index), so that none of this stays live across the MFMA loop
    int tid = int(threadIdx.x);
    asm volatile("" : "+v"(tid));
    const int nq = a.nq;
    const int rowlen = a.BI[2] * nq;
    const int rpp = kThreads / rowlen;
    const int r0 = tid / rowlen;
    if (r0 >= rpp) return;
    const int cu = tid - r0 * rowlen;
    const int x = cu / nq, q = cu - x * nq;
    const int64_t t2 = i0[2] + x;
    const int c = c0 + q * kPerUnit;
    const int64_t vb = a.cin * esz;
    // the column's buffer, its W extent and the column's W coordinate in it
    const char* src = a.tile;
    int64_t e2 = a.P[2], u2 = t2;
    int64_t lok = 0, hik = 0;
    const char *slo = nullptr, *shi = nullptr;
    if constexpr (FK >= 0) {
        lok = a.fold.lo[FK];
        hik = lok + a.fold.ext[FK];
        slo = a.fold.slab[FK][0];
        shi = a.fold.slab[FK][1];
    }
    if constexpr (FK == 2) {
        const bool lo = t2 < lok, hi = t2 >= hik;
        src = lo ? slo : (hi ? shi : a.tile);
        e2 = lo ? lok : (hi ? a.P[2] - hik : a.P[2]);
        u2 = hi ? t2 - hik : t2;
    }
    const bool colok = t2 >= 0 && t2 < a.P[2] && c < a.cin && src != nullptr;
    // rows z of the brick with i0[0] + z inside the tile are [zlo, zhi); same for y
    const int BI0 = a.BI[0], BI1 = a.BI[1];
    const int zlo = int(std::min<int64_t>(std::max<int64_t>(-i0[0], 0), BI0));
    const int zhi = int(std::min<int64_t>(std::max<int64_t>(a.P[0] - i0[0], 0), BI0));
    const int ylo = int(std::min<int64_t>(std::max<int64_t>(-i0[1], 0), BI1));
    const int yhi = int(std::min<int64_t>(std::max<int64_t>(a.P[1] - i0[1], 0), BI1));
    // byte offset of unit (z, y) of the column in its buffer:
    // ((nn P0 + i0[0] + z) P1 + i0[1] + y) rowb + colb
    const int64_t rowb = e2 * vb, colb = u2 * vb + int64_t(c) * esz;
    const int dz = rpp / BI1, dy = rpp - dz * BI1;
    int z = r0 / BI1, y = r0 - z * BI1;
    int64_t off = ((nn * a.P[0] + i0[0] + z) * a.P[1] + i0[1] + y) * rowb + colb;
    const int64_t step = (int64_t(dz) * a.P[1] + dy) * rowb, wrap = (a.P[1] - BI1) * rowb;
    const int rows = BI0 * BI1;
    const int dstep = rpp * a.BI[2];
    uint4* dst = lds + q * nvp + r0 * a.BI[2] + x;
    for (int r = r0; r < rows; r += B * rpp) {
        uint4 val[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            val[j] = make_uint4(0, 0, 0, 0);
            if (r + j * rpp < rows && colok && z >= zlo && z < zhi && y >= ylo && y < yhi) {
                if constexpr (FK == 0 || FK == 1) {
                    // the row's buffer: the row index in it times the row bytes
                    const int64_t t0 = i0[0] + z, t1 = i0[1] + y;
                    const int64_t tk = FK == 0 ? t0 : t1;
                    const bool lo = tk < lok, hi = tk >= hik;
                    const char* base = lo ? slo : (hi ? shi : a.tile);
                    const int64_t ek = lo ? lok : (hi ? a.P[FK] - hik : a.P[FK]);
                    const int64_t ck = hi ? tk - hik : tk;
                    const int64_t row = FK == 0 ? (nn * ek + ck) * a.P[1] + t1 : (nn * a.P[0] + t0) * ek + ck;
                    if (base) val[j] = *reinterpret_cast<const uint4*>(base + row * rowb + colb);
                } else {
                    val[j] = *reinterpret_cast<const uint4*>(src + off);
                }
            }
            z += dz;
            y += dy;
            off += step;
            if (y >= BI1) {
                y -= BI1;
                ++z;
                off += wrap;
            }
        }
#pragma unroll
        for (int j = 0; j < B; ++j)
            if (r + j * rpp < rows) dst[j * dstep] = val[j];
        dst += B * dstep;
    }
}

// Stage the input brick channels [c0, c0 + cc) into LDS; SB units in flight
// per thread on the row paths.
template <typename T, int SB>
__device__ __forceinline__ void stage_brick(const FwdArgs& a, uint4* lds, int64_t nn, const int64_t i0[3], int c0)
{
    constexpr int kPerUnit = 16 / Traits<T>::esz;
    const bool vec_ok = a.vec != 0;
    const int nvp = a.BI[0] * a.BI[1] * a.BI[2];  // voxels per unit plane
    // a brick whose footprint (clipped to the tile) stays off every folded
    // margin reads the tile alone: the plain loads below
    bool margin = false;
    for (int k = 0; k < 3; ++k) {
        if (!((a.fold.mask >> k) & 1u)) continue;
        const int64_t f0 = i0[k] > 0 ? i0[k] : 0;
        const int64_t f1 = i0[k] + a.BI[k] < a.P[k] ? i0[k] + a.BI[k] : a.P[k];
        margin = margin || (f0 < f1 && (f0 < a.fold.lo[k] || f1 > a.fold.lo[k] + a.fold.ext[k]));
    }
    const uint32_t fm = a.fold.mask;
    const bool rows_ok = vec_ok && a.cin % kPerUnit == 0 && a.BI[2] * a.nq <= kThreads;
    if (margin && rows_ok && (fm == 1u || fm == 2u || fm == 4u)) {
        if (fm == 1u)
            stage_rows<T, SB, 0>(a, lds, nvp, nn, i0, c0);
        else if (fm == 2u)
            stage_rows<T, SB, 1>(a, lds, nvp, nn, i0, c0);
        else
            stage_rows<T, SB, 2>(a, lds, nvp, nn, i0, c0);
        return;
    }
    if (margin && (fm == 1u || fm == 2u || fm == 4u)) {
        // margins on one axis k: a voxel comes from the tile, or from the slab
        // of its side, whose layout is the tile's with axis k cut to the margin
        const int k = fm == 1u ? 0 : (fm == 2u ? 1 : 2);
        const int64_t lok = a.fold.lo[k], hik = a.fold.lo[k] + a.fold.ext[k], Pk = a.P[k];
        const char* slo = a.fold.slab[k][0];
        const char* shi = a.fold.slab[k][1];
        const int64_t vb = a.cin * Traits<T>::esz;
        stage_units(a, lds, nvp, [&](int v, int q, int z, int y, int x) {
            const int64_t t0 = i0[0] + z, t1 = i0[1] + y, t2 = i0[2] + x;
            const int c = c0 + q * kPerUnit;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] && c < a.cin) {
                const int64_t tk = k == 0 ? t0 : (k == 1 ? t1 : t2);
                const bool lo = tk < lok, hi = tk >= hik;
                const char* base = lo ? slo : (hi ? shi : a.tile);
                const int64_t ek = lo ? lok : (hi ? Pk - hik : Pk);
                const int64_t ck = hi ? tk - hik : tk;
                const int64_t e1 = k == 1 ? ek : a.P[1], e2 = k == 2 ? ek : a.P[2];
                const int64_t d0 = k == 0 ? ek : a.P[0];
                const int64_t u0 = k == 0 ? ck : t0, u1 = k == 1 ? ck : t1, u2 = k == 2 ? ck : t2;
                if (base) {
                    const T* src = reinterpret_cast<const T*>(base + (((nn * d0 + u0) * e1 + u1) * e2 + u2) * vb) + c;
                    if (vec_ok && c + kPerUnit <= a.cin) {
                        val = *reinterpret_cast<const uint4*>(src);
                    } else {
                        T tmp[kPerUnit];
#pragma unroll
                        for (int e = 0; e < kPerUnit; ++e) tmp[e] = (c + e < a.cin) ? src[e] : T(0);
                        val = *reinterpret_cast<const uint4*>(tmp);
                    }
                }
            }
            return val;
        });
        return;
    }
    if (margin) {
        // margin voxels come from the received slabs (or are zero)
        stage_units(a, lds, nvp, [&](int v, int q, int z, int y, int x) {
            const int64_t t0 = i0[0] + z, t1 = i0[1] + y, t2 = i0[2] + x;
            const int c = c0 + q * kPerUnit;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] && c < a.cin) {
                const char* vox = fold_voxel(a.fold, a.tile, nn, t0, t1, t2, a.cin * Traits<T>::esz);
                if (vox) {
                    const T* src = reinterpret_cast<const T*>(vox) + c;
                    if (vec_ok && c + kPerUnit <= a.cin) {
                        val = *reinterpret_cast<const uint4*>(src);
                    } else {
                        T tmp[kPerUnit];
#pragma unroll
                        for (int e = 0; e < kPerUnit; ++e) tmp[e] = (c + e < a.cin) ? src[e] : T(0);
                        val = *reinterpret_cast<const uint4*>(tmp);
                    }
                }
            }
            return val;
        });
        return;
    }
    if (rows_ok) {
        stage_rows<T, SB, -1>(a, lds, nvp, nn, i0, c0);
        return;
    }
    stage_units(a, lds, nvp, [&](int v, int q, int z, int y, int x) {
        const int64_t t0 = i0[0] + z, t1 = i0[1] + y, t2 = i0[2] + x;
        const int c = c0 + q * kPerUnit;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] && c < a.cin) {
            const int64_t off = ((((nn * a.P[0] + t0) * a.P[1] + t1) * a.P[2] + t2) * a.cin + c) * Traits<T>::esz;
            if (vec_ok && c + kPerUnit <= a.cin) {
                val = *reinterpret_cast<const uint4*>(a.tile + off);
            } else {
                T tmp[kPerUnit];
                const T* src = reinterpret_cast<const T*>(a.tile + off);
#pragma unroll
                for (int e = 0; e < kPerUnit; ++e) tmp[e] = (c + e < a.cin) ? src[e] : T(0);
                val = *reinterpret_cast<const uint4*>(tmp);
            }
        }
        return val;
    });
}

template <typename T>
__device__ __forceinline__ void mfma_step(f32x16_t& acc, uint4 av, uint4 bv);

template <>
__device__ __forceinline__ void mfma_step<bf16_t>(f32x16_t& acc, uint4 av, uint4 bv)
{
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv),
                                                   acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_step<float>(f32x16_t& acc, uint4 av, uint4 bv)
{
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av.x), __uint_as_float(bv.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av.y), __uint_as_float(bv.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av.z), __uint_as_float(bv.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(av.w), __uint_as_float(bv.w), acc, 0, 0, 0);
}

// Brick b (in the XCD-aware order) of one region.
template <typename T, int RM, int RN>
__device__ __forceinline__ void fwd_tiled_body(const FwdArgs& a, int64_t b)
{
    extern __shared__ uint4 lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int row = lane & 31;

    // block -> (n, brick, N group)
    const int ngi = int(b % a.ng);
    b /= a.ng;
    const int bx = int(b % a.NB[2]);
    b /= a.NB[2];
    const int by = int(b % a.NB[1]);
    b /= a.NB[1];
    const int bz = int(b % a.NB[0]);
    const int64_t nn = b / a.NB[0];
    const int64_t ob[3] = {int64_t(bz) * a.BO[0], int64_t(by) * a.BO[1], int64_t(bx) * a.BO[2]};
    const int64_t i0[3] = {(a.org[0] + ob[0]) * a.S[0] - a.pad[0], (a.org[1] + ob[1]) * a.S[1] - a.pad[1],
                           (a.org[2] + ob[2]) * a.S[2] - a.pad[2]};
    const int nt0 = ngi * RN;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];

    // per-lane LDS voxel base of each of this wave's M tiles. A-row `row` of a
    // tile holds brick voxel tile*32 + row, or with rperm (8-voxel brick rows)
    // voxel tile*32 + 8 (row % 4) + row / 4: the 16 lanes that the LDS serves
    // together then read four brick rows, which spreads them over the banks
    const int prow = a.rperm ? 8 * (row & 3) + (row >> 2) : row;
    int vbase[RM];
#pragma unroll
    for (int i = 0; i < RM; ++i) {
        const int f = (wave * RM + i) * 32 + prow;
        const int ff = f < bov ? f : 0;
        const int ox = ff % a.BO[2];
        const int oy = (ff / a.BO[2]) % a.BO[1];
        const int oz = ff / (a.BO[2] * a.BO[1]);
        vbase[i] = (oz * a.S[0] * a.BI[1] + oy * a.S[1]) * a.BI[2] + ox * a.S[2];
    }

    f32x16_t acc[RM][RN];
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int taps = a.K[0] * a.K[1] * a.K[2];
    const int kcp = a.cc / Traits<T>::kc;  // K-chunks per pass
    const int plane = a.BI[1] * a.BI[2];
    for (int p = 0; p < a.npass; ++p) {
        if (p > 0) __syncthreads();
        stage_brick<T, kStageBatch>(a, lds, nn, i0, p * a.cc);
        __syncthreads();
        const int iters = taps * kcp;
        // Iteration = (tap, channel chunk). Software pipeline over two operand
        // sets that alternate (no register copies): the A fragments (LDS) and B
        // fragments (weights, L2) of iteration it + 1 are in flight while
        // iteration it multiplies; every load is unconditional (the one past the
        // last iteration re-reads the last, in bounds), so the waits before each
        // set's MFMAs cover exactly that set's loads.
        // The iteration state is advanced by uniform increments (scalar
        // registers): the weight fragments' base moves by one K-chunk per
        // iteration and skips the other passes' chunks at the end of a tap;
        // the tap's brick offset moves by one voxel, and by the rest of a row
        // or plane where kw or kh wraps. A lane adds only its own offsets.
        struct TapIt {
            const uint4* b;  // fragment (tap, chunk) of N tile nt0
            int toff;        // brick voxel offset of the tap
            int kc, t2, t1;
        };
        const int64_t ks = int64_t(a.nt) * 64;                 // one K-chunk
        const int64_t ts = int64_t(a.nkc - kcp) * a.nt * 64;  // the other passes' chunks
        const int wrap2 = a.BI[2] - a.K[2], wrap1 = plane - a.K[1] * a.BI[2];
        auto step_tap = [&](TapIt& s) {
            s.b += ks;
            if (++s.kc == kcp) {
                s.kc = 0;
                s.b += ts;
                ++s.toff;
                if (++s.t2 == a.K[2]) {
                    s.t2 = 0;
                    s.toff += wrap2;
                    if (++s.t1 == a.K[1]) {
                        s.t1 = 0;
                        s.toff += wrap1;
                    }
                }
            }
        };
        // the A fragment's byte address: unit plane 2 kc + g, voxel
        // vbase + toff; the lane's part is fixed, the rest uniform
        const char* ldsb = reinterpret_cast<const char*>(lds);
        const uint32_t plane16 = uint32_t(a.BI[0] * a.BI[1] * a.BI[2]) * 16u;
        uint32_t abase[RM];
#pragma unroll
        for (int i = 0; i < RM; ++i) abase[i] = uint32_t(g) * plane16 + uint32_t(vbase[i]) * 16u;
        auto load = [&](const TapIt& s, uint4 (&av)[RM], uint4 (&bv)[RN]) {
#pragma unroll
            for (int j = 0; j < RN; ++j) bv[j] = s.b[j * 64 + lane];
            const uint32_t u = uint32_t(2 * s.kc) * plane16 + uint32_t(s.toff) * 16u;
#pragma unroll
            for (int i = 0; i < RM; ++i) av[i] = *reinterpret_cast<const uint4*>(ldsb + (abase[i] + u));
        };
        auto mma = [&](const uint4 (&av)[RM], const uint4 (&bv)[RN]) {
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int j = 0; j < RN; ++j) mfma_step<T>(acc[i][j], av[i], bv[j]);
        };
        TapIt nx{a.wfrag + (int64_t(p) * kcp * a.nt + nt0) * 64, 0, 0, 0, 0};
        uint4 a0[RM], b0[RN], a1[RM], b1[RN];
        load(nx, a0, b0);
        int it = 0;
        for (; it + 1 < iters; it += 2) {
            step_tap(nx);
            load(nx, a1, b1);  // iteration it + 1
            mma(a0, b0);
            if (it + 2 < iters) step_tap(nx);
            load(nx, a0, b0);  // iteration it + 2 (past the end: it + 1 again)
            mma(a1, b1);
        }
        if (it < iters) mma(a0, b0);
    }

    // epilogue: lane holds column lane%32, rows 8*(r/4) + 4*g + (r%4). The
    // brick's output origin and the extents left from it, formed once
    T* y = reinterpret_cast<T*>(a.y) + a.ybase + nn * a.ys[0] + (a.org[0] + ob[0]) * a.ys[1] +
           (a.org[1] + ob[1]) * a.ys[2] + (a.org[2] + ob[2]) * a.ys[3];
    const int rem0 = int(a.O[0] - ob[0]), rem1 = int(a.O[1] - ob[1]), rem2 = int(a.O[2] - ob[2]);
    const int64_t ys1 = a.ys[1], ys2 = a.ys[2], ys3 = a.ys[3];
    const int cout_left = int(std::min<int64_t>(a.cout - int64_t(nt0) * 32, int64_t(RN) * 32));
    T* const ycol = y + int64_t(nt0) * 32;
    if (a.yvec) {
        // Through LDS, one 32 x 32 tile at a time in a region of the wave's own
        // (the brick is no longer read once every wave is past the barrier):
        // the lanes write their elements, then each lane stores whole 16-byte
        // runs of output channels of one voxel. Brick coordinates of a lane's
        // rows advance by carries from one division per tile.
        __syncthreads();
        constexpr int VE = 16 / int(sizeof(T));  // elements per 16 bytes
        constexpr int CPR = 32 / VE;             // 16-byte runs per tile row
        constexpr int RSTEP = 64 / CPR;          // rows between a lane's runs
        T* tl = reinterpret_cast<T*>(lds) + wave * 32 * 32;
        const int crow = lane / CPR, ccol = (lane % CPR) * VE;
#pragma unroll
        for (int i = 0; i < RM; ++i) {
            const int f0 = (wave * RM + i) * 32 + crow;
            int ox0 = f0 % a.BO[2], oy0 = (f0 / a.BO[2]) % a.BO[1], oz0 = f0 / (a.BO[2] * a.BO[1]);
#pragma unroll
            for (int j = 0; j < RN; ++j) {
                // accumulator row 8 (r / 4) + 4 g + r % 4 is brick voxel tile*32 + that
                // row, or (rperm) tile*32 + 8 (r % 4) + 2 (r / 4) + g; the LDS tile is
                // indexed by voxel
                if (a.rperm) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        tl[(8 * (r & 3) + 2 * (r >> 2) + g) * 32 + (lane & 31)] = from_f32<T>(acc[i][j][r]);
                } else {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        tl[(8 * (r >> 2) + 4 * g + (r & 3)) * 32 + (lane & 31)] = from_f32<T>(acc[i][j][r]);
                }
                // a wave's LDS accesses complete in issue order: its reads
                // below see its writes above, and the next tile's writes come
                // after these reads
                int ox = ox0, oy = oy0, oz = oz0;
#pragma unroll
                for (int k = 0; k < 32 / RSTEP; ++k) {
                    if (k > 0) {
                        ox += RSTEP;
                        while (ox >= a.BO[2]) {
                            ox -= a.BO[2];
                            if (++oy == a.BO[1]) {
                                oy = 0;
                                ++oz;
                            }
                        }
                    }
                    const int row = crow + k * RSTEP;
                    const uint4 v = *reinterpret_cast<const uint4*>(tl + row * 32 + ccol);
                    const int f = f0 + k * RSTEP;
                    const int co = j * 32 + ccol;
                    // nontemporal: the outputs are not read again by this kernel
                    if (f < bov && oz < rem0 && oy < rem1 && ox < rem2 && co < cout_left)
                        __builtin_nontemporal_store(__builtin_bit_cast(lds_u32x4, v),
                                                    reinterpret_cast<lds_u32x4*>(ycol + oz * ys1 + oy * ys2 +
                                                                                 ox * ys3 + co));
                }
            }
        }
        return;
    }
    // otherwise element by element; the brick coordinates of a row are
    // advanced from the previous row's (carries instead of divisions)
#pragma unroll
    for (int i = 0; i < RM; ++i) {
        const int fb = (wave * RM + i) * 32 + 4 * g;
        int ox = fb % a.BO[2];
        int oy = (fb / a.BO[2]) % a.BO[1];
        int oz = fb / (a.BO[2] * a.BO[1]);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if (r > 0) {
                ox += (r & 3) == 0 ? 5 : 1;
                while (ox >= a.BO[2]) {
                    ox -= a.BO[2];
                    if (++oy == a.BO[1]) {
                        oy = 0;
                        ++oz;
                    }
                }
            }
            const int f = fb + 8 * (r >> 2) + (r & 3);
            if (f >= bov) continue;
            if (oz >= rem0 || oy >= rem1 || ox >= rem2) continue;
            T* const yv = ycol + oz * ys1 + oy * ys2 + ox * ys3;
#pragma unroll
            for (int j = 0; j < RN; ++j) {
                const int co = j * 32 + row;
                if (co < cout_left) yv[co] = from_f32<T>(acc[i][j][r]);
            }
        }
    }
}

template <typename T, int RM, int RN>
__global__ __launch_bounds__(kThreads, 2) void conv_fwd_tiled(FwdArgs a)
{
    fwd_tiled_body<T, RM, RN>(a, xcd_remap(blockIdx.x, a.nblocks));
}

// Several regions in one launch: each takes its own inlined copy of the body,
// so that its arguments are read from a fixed place.
template <typename T, int RM, int RN>
__global__ __launch_bounds__(kThreads, 2) void conv_fwd_tiledn(FwdLaunch la)
{
    const int64_t b = xcd_remap(blockIdx.x, gridDim.x);
    if (b < la.end[0])
        fwd_tiled_body<T, RM, RN>(la.r[0], b);
    else if (b < la.end[1])
        fwd_tiled_body<T, RM, RN>(la.r[1], b - la.end[0]);
    else if (b < la.end[2])
        fwd_tiled_body<T, RM, RN>(la.r[2], b - la.end[1]);
    else
        fwd_tiled_body<T, RM, RN>(la.r[3], b - la.end[2]);
}

// wfrag[((tap * nkc + kc) * nt + ntile) * 64 + lane] = 16 bytes of weights in
// MFMA B-fragment order (see the file comment); zero past cin / cout.
template <typename T>
__global__ __launch_bounds__(256) void wfrag_kernel(const T* w, uint4* wfrag, int64_t cin, int64_t cout, int taps,
                                                    int nkc, int nt)
{
    constexpr int kPer = 16 / Traits<T>::esz;
    const int64_t total = int64_t(taps) * nkc * nt * 64;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        const int lane = int(e % 64);
        int64_t r = e / 64;
        const int ntile = int(r % nt);
        r /= nt;
        const int kc = int(r % nkc);
        const int tap = int(r / nkc);
        const int64_t co = int64_t(ntile) * 32 + (lane & 31);
        const int g = lane >> 5;
        T vals[kPer];
#pragma unroll
        for (int s = 0; s < kPer; ++s) {
            const int64_t ci = int64_t(kc) * Traits<T>::kc + g * kPer + s;
            vals[s] = (co < cout && ci < cin) ? w[(co * cin + ci) * taps + tap] : T(0);
        }
        wfrag[e] = *reinterpret_cast<const uint4*>(vals);
    }
}

template <typename T>
PlanF plan_fwd_t(const Tile3& t, const Conv3& cv, const int64_t* oext = nullptr, int64_t fix_cc = 0,
                 int rm_over = 0)
{
    // oext: the extent of the outputs to compute (a region; default the whole
    // box); fix_cc: a channel pass width to keep (a region's outputs are then
    // summed in the same order as in the whole box's plan: the order depends
    // on the passes, not on the tile shape); rm_over: M tiles per wave
    PlanF pl{};
    const int64_t O[3] = {oext ? oext[0] : cv.O[0], oext ? oext[1] : cv.O[1], oext ? oext[2] : cv.O[2]};
    constexpr int kc = Traits<T>::kc;
    constexpr int esz = Traits<T>::esz;
    const int64_t nt = ceil_div(cv.cout, 32);
    int rn, rm;
    if (std::is_same<T, bf16_t>::value) {
        rn = nt >= 2 ? 2 : 1;
        rm = rm_over == 2 && rn == 2 ? 2 : 4;
    } else {
        rn = nt >= 4 ? 4 : (nt >= 2 ? 2 : 1);
        rm = rn == 4 ? 1 : (rn == 2 ? 2 : 4);
    }
    const int64_t cap = int64_t(kWaves) * rm * 32;
    const int64_t cfull = round_up(t.c, kc);
    const size_t kLdsPref = 80 * 1024, kLdsMax = 160 * 1024;

    double best = 1e300;
    FwdArgs bestA{};
    size_t bestLds = 0;
    auto consider = [&](int64_t b0, int64_t b1, int64_t b2) {
        if (b0 < 1 || b1 < 1 || b2 < 1 || b0 * b1 * b2 > cap) return;
        int64_t bi[3], bo[3] = {b0, b1, b2};
        int64_t biv = 1;
        for (int k = 0; k < 3; ++k) {
            bi[k] = (bo[k] - 1) * cv.S[k] + cv.K[k];
            biv *= bi[k];
        }
        // channel pass width: the largest multiple of kc whose brick fits
        int64_t cc = cfull;
        if (fix_cc > 0)
            cc = fix_cc;
        else
            while (cc > kc && size_t(biv * cc * esz) > kLdsPref) cc = round_up(cc / 2, kc);
        size_t lds = size_t(biv * cc * esz);
        if (lds > kLdsMax) return;
        double eff = double(b0 * b1 * b2) / double(cap);
        for (int k = 0; k < 3; ++k) {
            const int64_t nb = ceil_div(O[k], bo[k]);
            eff *= double(O[k]) / double(nb * bo[k]);
        }
        double cost = double(biv) / double(b0 * b1 * b2) / eff;
        if (lds > kLdsPref) cost *= 1.5;
        cost *= 1.0 + 0.02 * double(ceil_div(cfull, cc) - 1);
        if (cost < best) {
            best = cost;
            bestLds = lds;
            FwdArgs a{};
            for (int k = 0; k < 3; ++k) {
                a.BO[k] = int32_t(bo[k]);
                a.BI[k] = int32_t(bi[k]);
                a.NB[k] = int32_t(ceil_div(cv.O[k], bo[k]));
            }
            a.cc = int32_t(cc);
            bestA = a;
        }
    };
    for (int64_t b2 = 1; b2 <= cap; b2 *= 2) {
        const int64_t w2 = std::min(b2, O[2]);
        for (int64_t b1 = 1; b1 * w2 <= cap; b1 *= 2) {
            const int64_t w1 = std::min(b1, O[1]);
            const int64_t w0 = std::min(cap / (w1 * w2), O[0]);
            consider(w0, w1, w2);
            for (int64_t b0 = 1; b0 < w0; b0 *= 2) consider(b0, w1, w2);
        }
    }
    if (best >= 1e299) return pl;
    FwdArgs& a = bestA;
    a.n = t.n;
    a.cin = t.c;
    a.cout = cv.cout;
    for (int k = 0; k < 3; ++k) {
        a.P[k] = t.P[k];
        a.O[k] = cv.O[k];
        a.K[k] = int32_t(cv.K[k]);
        a.S[k] = int32_t(cv.S[k]);
        a.pad[k] = int32_t(cv.pad[k]);
    }
    a.nq = int32_t(a.cc * esz / 16);
    a.npass = int32_t(ceil_div(cfull, a.cc));
    // fragment counts cover every index the kernel forms: npass * (cc / kc)
    // K-chunks and ng * rn N tiles; the padding holds zero weights
    a.nkc = int32_t(int64_t(a.npass) * (a.cc / kc));
    a.ng = int32_t(ceil_div(nt, rn));
    a.nt = int32_t(int64_t(a.ng) * rn);
    a.nblocks = t.n * int64_t(a.NB[0]) * a.NB[1] * a.NB[2] * a.ng;
    pl.rm = rm;
    pl.rn = rn;
    pl.a = a;
    pl.lds = bestLds;
    pl.ok = a.nblocks > 0 && a.nblocks < (int64_t(1) << 31);
    return pl;
}

bool tiled_supported(const Tile3& t, const Conv3& cv)
{
    // int32 LDS/brick indexing and per-axis sizes; the host planner checks LDS.
    for (int k = 0; k < 3; ++k)
        if (cv.K[k] > 64 || cv.S[k] > 64 || cv.O[k] > (int64_t(1) << 30) || std::abs(cv.pad[k]) > (1 << 29))
            return false;
    return t.c <= 4096 && cv.cout <= 4096;
}

template <typename T>
size_t wfrag_bytes(const Tile3& t, const Conv3& cv)
{
    const PlanF pl = plan_fwd_t<T>(t, cv);
    if (!pl.ok) return 0;
    return size_t(cv.taps()) * size_t(pl.a.nkc) * size_t(pl.a.nt) * 64 * 16;
}

// n (1 to kMaxRegions) plans in one launch
template <typename T, int RM, int RN>
hipError_t launch_tiled(const PlanF* pl, int n, hipStream_t s)
{
    const void* fn = n > 1 ? reinterpret_cast<const void*>(&conv_fwd_tiledn<T, RM, RN>)
                           : reinterpret_cast<const void*>(&conv_fwd_tiled<T, RM, RN>);
    size_t lds = 0;
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        lds = std::max(lds, pl[i].lds);
        total += pl[i].a.nblocks;
    }
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
    if (total >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    if (n == 1) {
        FwdArgs a = pl[0].a;
        void* args[] = {&a};
        return hipLaunchKernel(fn, dim3(unsigned(total)), dim3(kThreads), args, lds, s);
    }
    FwdLaunch la{};
    int64_t acc = 0;
    for (int i = 0; i < kMaxRegions; ++i) {
        if (i < n) {
            la.r[i] = pl[i].a;
            acc += pl[i].a.nblocks;
        }
        if (i < kMaxRegions - 1) la.end[i] = acc;
    }
    void* args[] = {&la};
    return hipLaunchKernel(fn, dim3(unsigned(total)), dim3(kThreads), args, lds, s);
}

template <typename T>
hipError_t launch_tiled_plans(const PlanF* pl, int n, hipStream_t s)
{
    if (n < 1 || n > kMaxRegions) return hipErrorInvalidValue;
    for (int i = 1; i < n; ++i)
        if (pl[i].rm != pl[0].rm || pl[i].rn != pl[0].rn) return hipErrorNotSupported;
    const int rm = pl[0].rm, rn = pl[0].rn;
    if (rm == 4 && rn == 1) return launch_tiled<T, 4, 1>(pl, n, s);
    if (rm == 4 && rn == 2) return launch_tiled<T, 4, 2>(pl, n, s);
    if (rm == 2 && rn == 2) return launch_tiled<T, 2, 2>(pl, n, s);
    if (rm == 1 && rn == 4) return launch_tiled<T, 1, 4>(pl, n, s);
    return hipErrorInvalidValue;
}

// Whether the M-tile rows take brick voxels transposed. The A reads of an
// M tile put 32 brick voxels, four rows of 8 when the brick is 8 voxels wide,
// on 32 lanes, the rows BI2 voxels apart in LDS. Measured for 16-byte reads
// (cycles per wave instruction, 4 waves per CU): rows 10 apart 48 in order
// against 32 transposed, 12 apart 32 against 27, 14 apart 48 against 32; rows
// 8 apart (a dense brick) 27 in order, 32 transposed; odd distances and wider
// bricks gain nothing. In the kernel: rows 10 apart (C4's W-paired input
// gradient) 3.5 % faster; rows 12 apart (C4's forward) bank-conflict cycles
// 2.4 -> 0.12 per LDS-active cycle at the same matrix-core utilisation and
// time within 1 %.
bool rows_transposed(const FwdArgs& a)
{
    return a.BO[2] == 8 && a.S[2] == 1 && (a.BI[2] == 10 || a.BI[2] == 12);
}

// Whether every buffer the loads may read is 16-byte aligned.
bool loads_aligned(const void* tile, const Fold* fold)
{
    if (reinterpret_cast<uintptr_t>(tile) % 16 != 0) return false;
    if (fold)
        for (int k = 0; k < 3; ++k)
            for (int sd = 0; sd < 2; ++sd)
                if (reinterpret_cast<uintptr_t>(fold->slab[k][sd]) % 16 != 0) return false;
    return true;
}

bool dense_map(const Conv3& cv, const OutMap& om)
{
    const OutMap dm = dense_out(cv);
    return om.base == 0 && om.str[0] == dm.str[0] && om.str[1] == dm.str[1] && om.str[2] == dm.str[2] &&
           om.str[3] == dm.str[3];
}

// The plan of region rg of the output box, every argument filled in. A
// region smaller than the box takes bricks of its own shape with the box's
// channel passes, so that every output is summed in the same order whatever
// region computes it.
template <typename T>
PlanF plan_region(const Tile3& t, const Conv3& cv, const void* tile, void* y, const OutMap& om, const Region& rg,
                  const Fold* fold, void* ws)
{
    PlanF pl = plan_fwd_t<T>(t, cv);
    if (!pl.ok) return pl;
    if (rg.ext[0] != cv.O[0] || rg.ext[1] != cv.O[1] || rg.ext[2] != cv.O[2]) {
        auto same_passes = [&](const PlanF& q) {
            return q.ok && q.rn == pl.rn && q.a.cc == pl.a.cc && q.a.npass == pl.a.npass && q.a.nkc == pl.a.nkc &&
                   q.a.nt == pl.a.nt;
        };
        PlanF pr = plan_fwd_t<T>(t, cv, rg.ext, pl.a.cc);
        // a thin region with fewer bricks than the 512 resident workgroups
        // takes half-height bricks (two M tiles per wave) where that exists
        auto region_blocks = [&](const PlanF& q) {
            return t.n * ceil_div(rg.ext[0], q.a.BO[0]) * ceil_div(rg.ext[1], q.a.BO[1]) *
                   ceil_div(rg.ext[2], q.a.BO[2]) * q.a.ng;
        };
        if (same_passes(pr) && pr.rm == 4 && pr.rn == 2 && region_blocks(pr) < 512) {
            const PlanF p2 = plan_fwd_t<T>(t, cv, rg.ext, pl.a.cc, 2);
            if (same_passes(p2) && p2.rm == 2) pr = p2;
        }
        if (same_passes(pr)) pl = pr;
    }
    for (int k = 0; k < 3; ++k) {
        pl.a.O[k] = rg.ext[k];
        pl.a.NB[k] = int32_t(ceil_div(rg.ext[k], pl.a.BO[k]));
    }
    pl.a.nblocks = t.n * int64_t(pl.a.NB[0]) * pl.a.NB[1] * pl.a.NB[2] * pl.a.ng;
    pl.a.ybase = om.base;
    for (int k = 0; k < 4; ++k) {
        pl.a.ys[k] = om.str[k];
        if (k < 3) pl.a.org[k] = rg.org[k];
    }
    if (fold) pl.a.fold = *fold;
    pl.a.tile = static_cast<const char*>(tile);
    pl.a.vec = loads_aligned(tile, fold) && (t.c * Traits<T>::esz) % 16 == 0;
    {
        const int64_t ve = 16 / Traits<T>::esz;
        bool yv = reinterpret_cast<uintptr_t>(y) % 16 == 0 && cv.cout % ve == 0 && om.base % ve == 0;
        for (int k = 0; k < 4; ++k) yv = yv && om.str[k] % ve == 0;
        pl.a.yvec = yv ? 1 : 0;
    }
    pl.a.rperm = pl.a.yvec && rows_transposed(pl.a) ? 1 : 0;
    pl.a.wfrag = static_cast<const uint4*>(ws);
    pl.a.y = static_cast<char*>(y);
    return pl;
}

// Lay out the weight fragments of (t, cv) in ws; they depend on (t, cv) only,
// so a call over several regions lays them out once.
template <typename T>
hipError_t lay_wfrag(const Tile3& t, const Conv3& cv, const PlanF& pl, const void* w, void* ws, hipStream_t s)
{
    const int taps = int(cv.taps());
    const int64_t frag_total = int64_t(taps) * pl.a.nkc * pl.a.nt * 64;
    const unsigned fg = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(frag_total, 256), 4096)));
    hipLaunchKernelGGL(wfrag_kernel<T>, dim3(fg), dim3(256), 0, s, static_cast<const T*>(w), static_cast<uint4*>(ws),
                       t.c, cv.cout, taps, pl.a.nkc, pl.a.nt);
    return hipGetLastError();
}

template <typename T>
hipError_t run_fwd(const Tile3& t, const Conv3& cv, const void* tile, const void* w, void* y, const OutMap& om,
                   const Region& rg, const Fold* fold, bool rows, void* ws, bool frags_ready, hipStream_t s)
{
    const PlanF pl = plan_region<T>(t, cv, tile, y, om, rg, fold, ws);
    if (!pl.ok) return hipErrorInvalidValue;
    if (!frags_ready) {
        const hipError_t e = lay_wfrag<T>(t, cv, pl, w, ws, s);
        if (e != hipSuccess) return e;
    }
    if (rows)
        return launch_conv_fwd_rows(t, cv, std::is_same<T, bf16_t>::value ? SHARD_BF16 : SHARD_F32, tile, ws,
                                    pl.a.nkc, pl.a.nt, y, rg, fold, s);
    return launch_tiled_plans<T>(&pl, 1, s);
}

// n (2 to kMaxRegions) regions in one launch of the tiled kernel;
// hipErrorNotSupported, with nothing launched, when their plans take
// different kernels.
template <typename T>
hipError_t run_fwd_group(const Tile3& t, const Conv3& cv, const void* tile, const void* w, void* y, const OutMap& om,
                         const Region* rs, int n, const Fold* fold, void* ws, bool frags_ready, hipStream_t s)
{
    if (n < 2 || n > kMaxRegions) return hipErrorNotSupported;
    PlanF pl[kMaxRegions];
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        pl[i] = plan_region<T>(t, cv, tile, y, om, rs[i], fold, ws);
        if (!pl[i].ok) return hipErrorInvalidValue;
        if (pl[i].rm != pl[0].rm || pl[i].rn != pl[0].rn) return hipErrorNotSupported;
        total += pl[i].a.nblocks;
    }
    if (total >= (int64_t(1) << 31)) return hipErrorNotSupported;
    if (!frags_ready) {
        const hipError_t e = lay_wfrag<T>(t, cv, pl[0], w, ws, s);
        if (e != hipSuccess) return e;
    }
    return launch_tiled_plans<T>(pl, n, s);
}

}  // namespace

size_t generic_wgrad_workspace(const Tile3& t, const Conv3& cv);
hipError_t generic_conv_fwd(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* w,
                            void* y, const OutMap& om, const Region& rg, const Fold* fold, hipStream_t s);

OutMap dense_out(const Conv3& cv)
{
    OutMap m;
    m.base = 0;
    m.str[3] = cv.cout;
    m.str[2] = cv.O[2] * m.str[3];
    m.str[1] = cv.O[1] * m.str[2];
    m.str[0] = cv.O[0] * m.str[1];
    return m;
}

size_t conv_fwd_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    return dt == SHARD_BF16 ? wfrag_bytes<bf16_t>(t, cv) : wfrag_bytes<float>(t, cv);
}

FwdFamily fwd_family(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* y,
                     const OutMap& om, const Fold* fold, const void* ws)
{
    if (force_generic() || !tiled_supported(t, cv)) return FWD_GENERIC;
    const PlanF pl = dt == SHARD_BF16 ? plan_fwd_t<bf16_t>(t, cv) : plan_fwd_t<float>(t, cv);
    if (!pl.ok) return FWD_GENERIC;
    if (dense_map(cv, om) && conv_fwd_rows_supported(t, cv, dt, tile, ws, pl.a.nkc, pl.a.nt, y, fold))
        return FWD_ROWS;
    return FWD_TILED;
}

hipError_t launch_conv_fwd_region(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                  const void* w, void* y, const OutMap& om, const Region& rg, const Fold* fold,
                                  FwdFamily fam, void* ws, hipStream_t s, bool frags_ready)
{
    if (t.n * rg.ext[0] * rg.ext[1] * rg.ext[2] == 0) return hipSuccess;
    if (fam == FWD_GENERIC) return generic_conv_fwd(t, cv, dt, tile, w, y, om, rg, fold, s);
    const bool rows = fam == FWD_ROWS;
    return dt == SHARD_BF16 ? run_fwd<bf16_t>(t, cv, tile, w, y, om, rg, fold, rows, ws, frags_ready, s)
                            : run_fwd<float>(t, cv, tile, w, y, om, rg, fold, rows, ws, frags_ready, s);
}

hipError_t launch_conv_fwd_region_pair(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                       const void* w, void* y, const Region& ra, const Region& rb, const Fold* fold,
                                       void* ws, hipStream_t s, bool frags_ready)
{
    if (dt != SHARD_BF16) return hipErrorNotSupported;
    const PlanF pl = plan_fwd_t<bf16_t>(t, cv);
    if (!pl.ok || !conv_fwd_rows_supported(t, cv, dt, tile, ws, pl.a.nkc, pl.a.nt, y, fold))
        return hipErrorNotSupported;
    // the pair's own checks before anything is launched (the weight layout
    // included), so that a refusal leaves the stream untouched
    if (ra.org[2] != 0 || ra.ext[2] != cv.O[2] || rb.org[1] != ra.org[1] || rb.ext[1] != ra.ext[1] ||
        rb.org[2] != ra.org[2] || rb.ext[2] != ra.ext[2] ||
        (rb.org[0] < ra.org[0] + ra.ext[0] && ra.org[0] < rb.org[0] + rb.ext[0]) || t.c != 32)
        return hipErrorNotSupported;
    if (!frags_ready) {
        const int taps = int(cv.taps());
        const int64_t frag_total = int64_t(taps) * pl.a.nkc * pl.a.nt * 64;
        const unsigned fg = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(frag_total, 256), 4096)));
        hipLaunchKernelGGL(wfrag_kernel<bf16_t>, dim3(fg), dim3(256), 0, s, static_cast<const bf16_t*>(w),
                           static_cast<uint4*>(ws), t.c, cv.cout, taps, pl.a.nkc, pl.a.nt);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return launch_conv_fwd_rows(t, cv, dt, tile, ws, pl.a.nkc, pl.a.nt, y, ra, fold, s, &rb);
}

hipError_t launch_conv_fwd_tiled_group(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                       const void* w, void* y, const OutMap& om, const Region* rs, int n,
                                       const Fold* fold, void* ws, hipStream_t s, bool frags_ready)
{
    return dt == SHARD_BF16 ? run_fwd_group<bf16_t>(t, cv, tile, w, y, om, rs, n, fold, ws, frags_ready, s)
                            : run_fwd_group<float>(t, cv, tile, w, y, om, rs, n, fold, ws, frags_ready, s);
}

hipError_t launch_conv_fwd_mapped(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                  const void* w, void* y, const OutMap& om, void* ws, hipStream_t s)
{
    Region all{};
    for (int k = 0; k < 3; ++k) all.ext[k] = cv.O[k];
    const FwdFamily fam = fwd_family(t, cv, dt, tile, y, om, nullptr, ws);
    return launch_conv_fwd_region(t, cv, dt, tile, w, y, om, all, nullptr, fam, ws, s);
}

hipError_t launch_conv_fwd(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* w,
                           void* y, void* ws, hipStream_t s)
{
    return launch_conv_fwd_mapped(t, cv, dt, tile, w, y, dense_out(cv), ws, s);
}

}  // namespace shardconv
