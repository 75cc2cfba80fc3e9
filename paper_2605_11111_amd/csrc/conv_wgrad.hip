// Weight gradient of a shard on MFMA: dW[co][ci][t] = sum over the shard's
// output voxels v of dy[v][co] * tile[v*S + t - pad][ci].
//
// GEMM view: M = output channels, N = input channels (per tap), K = output
// voxels (millions). Split-K: the output bricks are cut into `nsplit`
// contiguous ranges; a workgroup sweeps one range for one channel block and
// tap group, keeps its dW tile in registers, and writes it once to the
// workspace; a reduce kernel sums the ranges in a fixed order (bit-identical
// results run to run, no atomics).
//
// bf16 (v_mfma_f32_16x16x32_bf16): each lane needs 8 consecutive K values
// (voxels) of one channel, so both operands are staged in LDS transposed,
// [channel][voxel]. Four waves own the 2x2 (or 4x1) 16x16 channel sub-tiles
// of a 32x32 (or 64x16) block; every wave sweeps all taps of its group. For
// tap (kd, kh, kw) a lane's 8 input voxels are 8 consecutive x positions
// shifted by kw: it reads the two aligned 16-byte blocks covering them once
// per (kd, kh) and derives every kw's operand with funnel shifts.
// fp32 (v_mfma_f32_32x32x2_f32): one K value per lane, so both operands come
// straight from channels-last LDS copies; the four waves split the taps.
#include <algorithm>
#include <cstdlib>
#include <utility>

#include "common.h"
#include "internal.h"

#define SC_LDSW(p) ((__attribute__((address_space(3))) void*)(p))

namespace shardconv {

size_t generic_wgrad_workspace(const Tile3& t, const Conv3& cv);
hipError_t generic_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                              float* dw, void* ws, const Fold* fold, hipStream_t s);

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_w;
typedef __attribute__((ext_vector_type(4))) float f32x4_w;
typedef __attribute__((ext_vector_type(16))) float f32x16_w;

namespace {

constexpr int kThreads = 256;
constexpr int kTargetBlocks = 512;  // two resident workgroups per CU on 256 CUs

// staging units rounded up to whole load instructions of the workgroup
__host__ __device__ inline int dl_round(int units) { return (units + kThreads - 1) / kThreads * kThreads; }

struct WgArgs {
    const char* tile;
    const char* dy;
    float* part;
    float* dw;
    int64_t n, cin, cout;
    int64_t P[3], O[3];
    int32_t K[3], S[3], pad[3];
    int32_t BO[3];
    int32_t NB[3];
    int64_t nbricks;
    int32_t nsplit, nmb, ncb, ntg;
    int32_t kdg;          // bf16: kd planes per tap group; fp32: taps per group
    int32_t biz, biy, bix, bixp;
    int32_t cs, csd;      // LDS channel strides (bf16 layout, elements)
    int32_t dy_off;       // byte offset of the dy copy in LDS
    int32_t blk;          // floats of partial dW per workgroup
    int32_t wco, wci;     // bf16: 16-wide sub-tiles per wave grid
    int32_t xvec, dvec;   // 16-byte vector loads allowed (alignment of base and channel rows)
    int64_t nblocks;
    Fold fold;            // halo folded into the loads when fold.mask != 0
    const char* zeros;    // 16 zero bytes in device memory (the status block's)
};

struct PlanW {
    int kind;  // 0 generic, 1 bf16 tiled, 2 fp32 tiled
    int kdg, k1, k2, wco;
    WgArgs a;
    size_t lds;
};

template <int S>
__device__ __forceinline__ uint4 funnel(const uint4& b0, const uint4& b1)
{
    const uint32_t w[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
    constexpr int d = S / 2;
    uint4 r;
    if constexpr (S % 2 == 0) {
        r.x = w[d];
        r.y = w[d + 1];
        r.z = w[d + 2];
        r.w = w[d + 3];
    } else {
        r.x = __builtin_amdgcn_alignbit(w[d + 1], w[d], 16);
        r.y = __builtin_amdgcn_alignbit(w[d + 2], w[d + 1], 16);
        r.z = __builtin_amdgcn_alignbit(w[d + 3], w[d + 2], 16);
        r.w = __builtin_amdgcn_alignbit(w[d + 4], w[d + 3], 16);
    }
    return r;
}

__device__ __forceinline__ void brick_origin(const WgArgs& a, int64_t br, int64_t& nn, int64_t ob[3])
{
    int64_t b = br;
    const int bx = int(b % a.NB[2]);
    b /= a.NB[2];
    const int by = int(b % a.NB[1]);
    b /= a.NB[1];
    const int bz = int(b % a.NB[0]);
    nn = b / a.NB[0];
    ob[0] = int64_t(bz) * a.BO[0];
    ob[1] = int64_t(by) * a.BO[1];
    ob[2] = int64_t(bx) * a.BO[2];
}

// Load 8 consecutive channels [c, c + 8) of one voxel (zeros past `cend`).
template <typename T>
__device__ __forceinline__ void load8(const T* src, int64_t c, int64_t cend, bool vec_ok, T out[8])
{
    if (vec_ok && c + 8 <= cend) {
        *reinterpret_cast<uint4*>(out) = *reinterpret_cast<const uint4*>(src);
        if constexpr (sizeof(T) == 4) *reinterpret_cast<uint4*>(out + 4) = *reinterpret_cast<const uint4*>(src + 4);
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) out[e] = (c + e < cend) ? src[e] : T(0);
    }
}

template <int KDG, int K1, int K2, int WCO>
__global__ __launch_bounds__(kThreads, 2) void wgrad_bf16_tiled(WgArgs a)
{
    constexpr int WCI = 4 / WCO;
    constexpr int TG = KDG * K1 * K2;
    constexpr int NCO = WCO * 16, NCI = WCI * 16;
    extern __shared__ uint4 lds4[];
    bf16_t* xs = reinterpret_cast<bf16_t*>(lds4);
    bf16_t* ds = reinterpret_cast<bf16_t*>(reinterpret_cast<char*>(lds4) + a.dy_off);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wco = wave / WCI, wci = wave % WCI;
    const int g = lane >> 4;
    const int l16 = lane & 15;

    int64_t b = xcd_remap(blockIdx.x, a.nblocks);
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    const int cb = int(b % a.ncb);
    b /= a.ncb;
    const int mb = int(b % a.nmb);
    const int64_t split = b / a.nmb;
    const int64_t br0 = split * a.nbricks / a.nsplit, br1 = (split + 1) * a.nbricks / a.nsplit;
    const int kd0 = tg * KDG;
    const int64_t co0 = int64_t(mb) * NCO, ci0 = int64_t(cb) * NCI;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    const bool xvec = a.xvec != 0;
    const bool dvec = a.dvec != 0;
    const bf16_t* tile = reinterpret_cast<const bf16_t*>(a.tile);
    const bf16_t* dy = reinterpret_cast<const bf16_t*>(a.dy);

    f32x4_w acc[TG];
#pragma unroll
    for (int i = 0; i < TG; ++i) acc[i] = f32x4_w{0.f, 0.f, 0.f, 0.f};

    for (int64_t br = br0; br < br1; ++br) {
        int64_t nn, ob[3];
        brick_origin(a, br, nn, ob);
        const int64_t i0 = ob[0] * a.S[0] + kd0 - a.pad[0];
        const int64_t i1 = ob[1] * a.S[1] - a.pad[1];
        const int64_t i2 = ob[2] - a.pad[2];
        __syncthreads();
        // X^T: [ci][z][y][x], zero outside the tile and past cin. A thread keeps
        // its (x, 8-channel unit) column and steps over (z, y) rows (one division
        // per row, none per unit) when a row of units fits the block.
        {
            const int rows = a.biz * a.biy;
            auto stage_x = [&](int q, int x, int row) {
                const int y = row % a.biy;
                const int z = row / a.biy;
                const int64_t t0 = i0 + z, t1 = i1 + y, t2 = i2 + x;
                const int64_t c = ci0 + 8 * q;
                bf16_t val[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                if (t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] && c < a.cin) {
                    const bf16_t* vox =
                        a.fold.mask ? reinterpret_cast<const bf16_t*>(fold_voxel(a.fold, a.tile, nn, t0, t1, t2,
                                                                                 a.cin * 2))
                                    : tile + (((nn * a.P[0] + t0) * a.P[1] + t1) * a.P[2] + t2) * a.cin;
                    if (vox) load8(vox + c, c, a.cin, xvec, val);
                }
                bf16_t* dst = xs + (8 * q) * a.cs + row * a.bixp + x;
#pragma unroll
                for (int e = 0; e < 8; ++e) dst[e * a.cs] = val[e];
            };
            constexpr int NQ = NCI / 8;
            const int rowlen = a.bix * NQ;
            if (rowlen <= kThreads) {
                const int rpp = kThreads / rowlen;
                const int r0 = int(threadIdx.x) / rowlen, cu = int(threadIdx.x) - r0 * rowlen;
                if (r0 < rpp)
                    for (int row = r0; row < rows; row += rpp) stage_x(cu % NQ, cu / NQ, row);
            } else {
                const int units = rows * rowlen;
                for (int u = threadIdx.x; u < units; u += kThreads) {
                    const int v = u / NQ;
                    stage_x(u % NQ, v % a.bix, v / a.bix);
                }
            }
        }
        // dy^T: [co][voxel of the output brick], zero past the output extent;
        // rows stepped as for X^T
        {
            auto stage_dy = [&](int q, int ox, int orow) {
                const int oy = orow % a.BO[1];
                const int oz = orow / a.BO[1];
                const int f = orow * a.BO[2] + ox;
                const int64_t o0 = ob[0] + oz, o1 = ob[1] + oy, o2 = ob[2] + ox;
                const int64_t c = co0 + 8 * q;
                bf16_t val[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                if (o0 < a.O[0] && o1 < a.O[1] && o2 < a.O[2] && c < a.cout)
                    load8(dy + (((nn * a.O[0] + o0) * a.O[1] + o1) * a.O[2] + o2) * a.cout + c, c, a.cout, dvec, val);
                bf16_t* dst = ds + (8 * q) * a.csd + f;
#pragma unroll
                for (int e = 0; e < 8; ++e) dst[e * a.csd] = val[e];
            };
            constexpr int NQ = NCO / 8;
            const int rowlen = a.BO[2] * NQ;
            const int orows = a.BO[0] * a.BO[1];
            if (rowlen <= kThreads) {
                const int rpp = kThreads / rowlen;
                const int r0 = int(threadIdx.x) / rowlen, cu = int(threadIdx.x) - r0 * rowlen;
                if (r0 < rpp)
                    for (int orow = r0; orow < orows; orow += rpp) stage_dy(cu % NQ, cu / NQ, orow);
            } else {
                const int units = orows * rowlen;
                for (int u = threadIdx.x; u < units; u += kThreads) {
                    const int f = u / NQ;
                    stage_dy(u % NQ, f % a.BO[2], f / a.BO[2]);
                }
            }
        }
        __syncthreads();
        const bf16_t* arow = ds + (wco * 16 + l16) * a.csd;
        const bf16_t* xrow = xs + (wci * 16 + l16) * a.cs;
        // the lane's 8 voxels [f0, f0 + 8) lie in one W row (BO[2] % 8 == 0);
        // their brick coordinates advance by carries as f0 steps by 32
        int ox0 = (8 * g) % a.BO[2], oy = ((8 * g) / a.BO[2]) % a.BO[1], oz = (8 * g) / (a.BO[2] * a.BO[1]);
        for (int ks = 0; ks < bov / 32; ++ks) {
            const int f0 = ks * 32 + 8 * g;
            if (ks > 0) {
                ox0 += 32;
                while (ox0 >= a.BO[2]) {
                    ox0 -= a.BO[2];
                    if (++oy == a.BO[1]) {
                        oy = 0;
                        ++oz;
                    }
                }
            }
            const uint4 av = *reinterpret_cast<const uint4*>(arow + f0);
#pragma unroll
            for (int kd = 0; kd < KDG; ++kd) {
#pragma unroll
                for (int kh = 0; kh < K1; ++kh) {
                    const bf16_t* src = xrow + ((oz * a.S[0] + kd) * a.biy + oy * a.S[1] + kh) * a.bixp + ox0;
                    const uint4 b0 = *reinterpret_cast<const uint4*>(src);
                    const uint4 b1 = K2 > 1 ? *reinterpret_cast<const uint4*>(src + 8) : b0;
#pragma unroll
                    for (int kw = 0; kw < K2; ++kw) {
                        uint4 bv;
                        if (kw == 0) bv = funnel<0>(b0, b1);
                        else if (kw == 1) bv = funnel<1>(b0, b1);
                        else if (kw == 2) bv = funnel<2>(b0, b1);
                        else if (kw == 3) bv = funnel<3>(b0, b1);
                        else if (kw == 4) bv = funnel<4>(b0, b1);
                        else if (kw == 5) bv = funnel<5>(b0, b1);
                        else if (kw == 6) bv = funnel<6>(b0, b1);
                        else bv = funnel<7>(b0, b1);
                        const int ti = (kd * K1 + kh) * K2 + kw;
                        acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                                          __builtin_bit_cast(bf16x8_w, bv), acc[ti],
                                                                          0, 0, 0);
                    }
                }
            }
        }
    }
    float4* out = reinterpret_cast<float4*>(a.part +
                                            ((((split * a.nmb + mb) * a.ncb + cb) * a.ntg + tg) * int64_t(a.blk)) +
                                            int64_t(wave) * TG * 256);
#pragma unroll
    for (int i = 0; i < TG; ++i) out[i * 64 + lane] = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
}

// bf16 with the staging of brick b + 1 in flight while brick b multiplies (a
// thread issues the global loads of its units of the next brick into registers
// before the brick's MFMAs and writes them to LDS after them), and the
// transposed LDS copies written four voxels at a time:
// a staging unit is four consecutive voxels (along W) of one 8-channel group,
// loaded as four 16-byte vectors into registers; after the brick's MFMAs each
// of its 8 channels is written as one 8-byte LDS store of the four voxels (the
// row-by-row 2-byte stores of wgrad_bf16_tiled cost eight stores per voxel
// and bank conflicts). LDS layouts, bricks, K steps and taps are those of
// wgrad_bf16_tiled: the partials are bit-identical. Units of the input brick
// run over (group of four x, channel group, row) with x fastest, units of dy
// over (quad of brick voxels, channel group), quads fastest: the lanes of a
// store instruction write consecutive 8-byte slots.
constexpr int kPipeBXU = 2;  // at most this many input staging units per thread
constexpr int kPipeBDU = 2;  // and dy staging units

template <int KDG, int K1, int K2, int WCO, int XU, int DU>
__global__ __launch_bounds__(kThreads, 2) void wgrad_bf16_pipe(WgArgs a)
{
    constexpr int WCI = 4 / WCO;
    constexpr int TG = KDG * K1 * K2;
    constexpr int NCO = WCO * 16, NCI = WCI * 16;
    constexpr int NQX = NCI / 8, NQD = NCO / 8;
    extern __shared__ uint4 lds4[];
    bf16_t* xs = reinterpret_cast<bf16_t*>(lds4);
    bf16_t* ds = reinterpret_cast<bf16_t*>(reinterpret_cast<char*>(lds4) + a.dy_off);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wco = wave / WCI, wci = wave % WCI;
    const int g = lane >> 4;
    const int l16 = lane & 15;

    int64_t b = xcd_remap(blockIdx.x, a.nblocks);
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    const int cb = int(b % a.ncb);
    b /= a.ncb;
    const int mb = int(b % a.nmb);
    const int64_t split = b / a.nmb;
    const int64_t br0 = split * a.nbricks / a.nsplit, br1 = (split + 1) * a.nbricks / a.nsplit;
    const int kd0 = tg * KDG;
    const int64_t co0 = int64_t(mb) * NCO, ci0 = int64_t(cb) * NCI;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    const bf16_t* tile = reinterpret_cast<const bf16_t*>(a.tile);
    const bf16_t* dy = reinterpret_cast<const bf16_t*>(a.dy);
    const int ngx = (a.bix + 3) / 4;             // groups of four x per input row
    const int nxu = a.biz * a.biy * ngx * NQX;   // input units
    const int ndu = (bov / 4) * NQD;             // dy units

    f32x4_w acc[TG];
#pragma unroll
    for (int i = 0; i < TG; ++i) acc[i] = f32x4_w{0.f, 0.f, 0.f, 0.f};

    uint4 xv[XU][4], dv[DU][4];
    auto issue = [&](int64_t br) {
        int64_t nn, ob[3];
        brick_origin(a, br, nn, ob);
        const int64_t i0 = ob[0] * a.S[0] + kd0 - a.pad[0];
        const int64_t i1 = ob[1] * a.S[1] - a.pad[1];
        const int64_t i2 = ob[2] - a.pad[2];
#pragma unroll
        for (int i = 0; i < XU; ++i) {
            const int u = tid + i * kThreads;
            const int gx = u % ngx, r = u / ngx;
            const int q = r % NQX, row = r / NQX;
            const int y = row % a.biy, z = row / a.biy;
            const int64_t t0 = i0 + z, t1 = i1 + y;
            const int64_t c = ci0 + 8 * q;
            const bool rowok = u < nxu && t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && c < a.cin;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int x = 4 * gx + j;
                const int64_t t2 = i2 + x;
                uint4 val = make_uint4(0u, 0u, 0u, 0u);
                if (rowok && x < a.bix && t2 >= 0 && t2 < a.P[2]) {
                    const bf16_t* vox =
                        a.fold.mask ? reinterpret_cast<const bf16_t*>(fold_voxel(a.fold, a.tile, nn, t0, t1, t2,
                                                                                 a.cin * 2))
                                    : tile + (((nn * a.P[0] + t0) * a.P[1] + t1) * a.P[2] + t2) * a.cin;
                    if (vox) val = *reinterpret_cast<const uint4*>(vox + c);
                }
                xv[i][j] = val;
            }
        }
#pragma unroll
        for (int i = 0; i < DU; ++i) {
            const int u = tid + i * kThreads;
            const int nq4 = bov / 4;
            const int f4 = u % nq4, q = u / nq4;
            const int f = 4 * f4;
            const int ox = f % a.BO[2];
            const int oy = (f / a.BO[2]) % a.BO[1];
            const int oz = f / (a.BO[2] * a.BO[1]);
            const int64_t o0 = ob[0] + oz, o1 = ob[1] + oy;
            const int64_t c = co0 + 8 * q;
            const bool rowok = u < ndu && o0 < a.O[0] && o1 < a.O[1] && c < a.cout;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t o2 = ob[2] + ox + j;
                uint4 val = make_uint4(0u, 0u, 0u, 0u);
                if (rowok && o2 < a.O[2])
                    val = *reinterpret_cast<const uint4*>(dy + (((nn * a.O[0] + o0) * a.O[1] + o1) * a.O[2] + o2) *
                                                                   a.cout + c);
                dv[i][j] = val;
            }
        }
    };
    // channel e of four voxels -> one 8-byte word (voxel j in bits 16 j ..)
    auto pick = [](const uint4 (&v)[4], int e) {
        auto half = [&](const uint4& w) {
            const uint32_t d = e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
            return (e & 1) ? (d >> 16) : (d & 0xFFFFu);
        };
        return make_uint2(half(v[0]) | (half(v[1]) << 16), half(v[2]) | (half(v[3]) << 16));
    };
    auto commit = [&]() {
#pragma unroll
        for (int i = 0; i < XU; ++i) {
            const int u = tid + i * kThreads;
            if (u < nxu) {
                const int gx = u % ngx, r = u / ngx;
                const int q = r % NQX, row = r / NQX;
                bf16_t* dst = xs + (8 * q) * a.cs + row * a.bixp + 4 * gx;
#pragma unroll
                for (int e = 0; e < 8; ++e) *reinterpret_cast<uint2*>(dst + e * a.cs) = pick(xv[i], e);
            }
        }
#pragma unroll
        for (int i = 0; i < DU; ++i) {
            const int u = tid + i * kThreads;
            if (u < ndu) {
                const int nq4 = bov / 4;
                const int f4 = u % nq4, q = u / nq4;
                bf16_t* dst = ds + (8 * q) * a.csd + 4 * f4;
#pragma unroll
                for (int e = 0; e < 8; ++e) *reinterpret_cast<uint2*>(dst + e * a.csd) = pick(dv[i], e);
            }
        }
    };

    if (br0 < br1) issue(br0);
    for (int64_t br = br0; br < br1; ++br) {
        __syncthreads();  // every wave is done reading the previous brick
        commit();
        __syncthreads();
        if (br + 1 < br1) issue(br + 1);
        const bf16_t* arow = ds + (wco * 16 + l16) * a.csd;
        const bf16_t* xrow = xs + (wci * 16 + l16) * a.cs;
        int ox0 = (8 * g) % a.BO[2], oy = ((8 * g) / a.BO[2]) % a.BO[1], oz = (8 * g) / (a.BO[2] * a.BO[1]);
        for (int ks = 0; ks < bov / 32; ++ks) {
            const int f0 = ks * 32 + 8 * g;
            if (ks > 0) {
                ox0 += 32;
                while (ox0 >= a.BO[2]) {
                    ox0 -= a.BO[2];
                    if (++oy == a.BO[1]) {
                        oy = 0;
                        ++oz;
                    }
                }
            }
            const uint4 av = *reinterpret_cast<const uint4*>(arow + f0);
            // input rows (kd, kh) of the K step, read LA rows ahead of their MFMAs
            constexpr int R = KDG * K1, LA = R < 3 ? R : 3;
            const bf16_t* src0 = xrow + ((oz * a.S[0]) * a.biy + oy * a.S[1]) * a.bixp + ox0;
            auto row_ptr = [&](int r) { return src0 + ((r / K1) * a.biy + (r % K1)) * a.bixp; };
            uint4 rb0[LA], rb1[LA];
#pragma unroll
            for (int r = 0; r < LA; ++r) {
                rb0[r] = *reinterpret_cast<const uint4*>(row_ptr(r));
                rb1[r] = K2 > 1 ? *reinterpret_cast<const uint4*>(row_ptr(r) + 8) : rb0[r];
            }
#pragma unroll
            for (int kd = 0; kd < KDG; ++kd) {
#pragma unroll
                for (int kh = 0; kh < K1; ++kh) {
                    const int r = kd * K1 + kh;
                    const uint4 b0 = rb0[r % LA];
                    const uint4 b1 = rb1[r % LA];
                    if (r + LA < R) {
                        rb0[r % LA] = *reinterpret_cast<const uint4*>(row_ptr(r + LA));
                        rb1[r % LA] = K2 > 1 ? *reinterpret_cast<const uint4*>(row_ptr(r + LA) + 8) : rb0[r % LA];
                    }
#pragma unroll
                    for (int kw = 0; kw < K2; ++kw) {
                        uint4 bv;
                        if (kw == 0) bv = funnel<0>(b0, b1);
                        else if (kw == 1) bv = funnel<1>(b0, b1);
                        else if (kw == 2) bv = funnel<2>(b0, b1);
                        else if (kw == 3) bv = funnel<3>(b0, b1);
                        else if (kw == 4) bv = funnel<4>(b0, b1);
                        else if (kw == 5) bv = funnel<5>(b0, b1);
                        else if (kw == 6) bv = funnel<6>(b0, b1);
                        else bv = funnel<7>(b0, b1);
                        const int ti = (kd * K1 + kh) * K2 + kw;
                        acc[ti] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                                          __builtin_bit_cast(bf16x8_w, bv), acc[ti],
                                                                          0, 0, 0);
                    }
                }
            }
        }
    }
    float4* out = reinterpret_cast<float4*>(a.part +
                                            ((((split * a.nmb + mb) * a.ncb + cb) * a.ntg + tg) * int64_t(a.blk)) +
                                            int64_t(wave) * TG * 256);
#pragma unroll
    for (int i = 0; i < TG; ++i) out[i * 64 + lane] = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
}

// Staging budget of the row-pair kernel below: load instructions per thread.
constexpr int kTrXU = 4;   // input
constexpr int kTrDU = 4;   // dy

// bf16, 16 input channels, one kd plane of taps per workgroup (the general
// kernel's decomposition for large 3D kernels such as 5 x 5 x 5): the row-pair
// kernel. No transposition while staging: the brick's input rows and dy are
// copied to LDS channels-last by direct global->LDS loads, and every operand is
// read with ds_read_b64_tr_b16 (lane i of a 16-lane group addresses voxel
// k0 + i / 4 at channels 4 (i % 4) ..; lane j receives channel j of voxels
// k0 .. k0 + 3). v_mfma_f32_32x32x16_bf16: M = 32 output channels (wave w owns
// channels 32 (w % 2) .. of the block's 64), K = 16 output voxels (one W run
// of the brick; lane k-half lane / 32 holds voxels 8 (lane / 32) ..), N = two
// taps of the 16 input channels: lane half h = (lane / 16) % 2 supplies columns
// 16 h .. of one tap. A tile is
//  * a row pair: taps (2 p + h, kw), 0 <= kw < K2, read from rows 2 p + h, or
//  * for odd K1, a W pair of the last row: taps (K1 - 1, 2 q + h), lane half h
//    reading the row one voxel further on (a tap past the kernel is computed
//    and dropped).
// Waves 0, 1 take the first ceil(T / 2) of the T tiles, waves 2, 3 the rest.
// Every lane addresses its own voxel rows, so a tile's B operand (voxels
// w .. w + 7 of its row, w = kw or 2 q) is two reads at voxel offsets w and
// w + 4 landing in the operand registers: no shuffles.
// LDS, per buffer: input voxel (z, y, x) of the brick at 32 (row rp + x), row =
// z biy + y, with a row pitch rp = 4 mod 8 voxels, so the two rows of a pair
// fall in opposite halves of the banks; dy voxel f at 128 f with its 32-byte
// channel chunk k at k ^ 2 ((f / 2) % 2). Two buffers: the loads of brick b + 1
// go out when brick b's compute starts, and one barrier per brick both
// publishes a brick and frees the other buffer. The operand reads of K step
// s + 1 are issued before the products of step s.
// The partials take the general kernel's layout; the sum over a K step is in
// a different order than there, so they match it to rounding, not bitwise.
template <int K1, int K2>
struct PrTiles {
    static_assert(K2 <= 5, "a 12-voxel run covers five W taps");
    static constexpr int NR = K1 / 2;                       // row-pair runs
    static constexpr int NW = K1 % 2 ? (K2 + 1) / 2 : 0;   // W-pair tiles
    static constexpr int T = NR * K2 + NW;
    static constexpr int NT0 = (T + 1) / 2;
    static constexpr int NRUN = NR + K1 % 2;
    static constexpr int run(int t) { return t < NR * K2 ? t / K2 : NR; }
    static constexpr int win(int t) { return t < NR * K2 ? t % K2 : 2 * (t - NR * K2); }
    static constexpr int kh(int t, int h) { return t < NR * K2 ? 2 * (t / K2) + h : K1 - 1; }
    static constexpr int kw(int t, int h) { return t < NR * K2 ? t % K2 : 2 * (t - NR * K2) + h; }
    static constexpr int first(int th) { return th == 0 ? 0 : NT0; }
    static constexpr int count(int th) { return th == 0 ? NT0 : T - NT0; }
    static constexpr bool uses(int th, int r)
    {
        for (int t = first(th); t < first(th) + count(th); ++t)
            if (run(t) == r) return true;
        return false;
    }
};

struct PrLayout {
    int rp, dy_off, bufb, bytes;
};

inline PrLayout pr_layout(const WgArgs& a)
{
    PrLayout L;
    L.rp = (a.bix + 3) / 4 * 4;
    if (L.rp % 8 == 0) L.rp += 4;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    L.dy_off = dl_round(a.biz * a.biy * L.rp * 2) * 16;
    L.bufb = L.dy_off + dl_round(bov * 8) * 16;
    L.bytes = 2 * L.bufb;
    return L;
}

// f(std::integral_constant<int, i>) for i = 0 .. N - 1, unrolled at compile time
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>)
{
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// one K step's operands: dy (A) and the input window of each of the wave's tiles
template <int NT>
struct PrOps {
    uint2 a[2];
    uint2 b[NT > 0 ? NT : 1][2];
};

template <int K1, int K2, int TH, bool FOLD>
__device__ __forceinline__ void wgrad_bf16_pr_body(const WgArgs& a, int rp, int dy_off, int bufb, uint32_t xbatch,
                                                   uint32_t dbatch)
{
    using TL = PrTiles<K1, K2>;
    constexpr int NT = TL::count(TH), T0 = TL::first(TH);
    constexpr int TG = K1 * K2;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int ch = wave & 1;
    const int li = lane & 15, vr = li >> 2;
    const int gh = (lane >> 4) & 1, gk = lane >> 5;

    int64_t b = xcd_remap(blockIdx.x, a.nblocks);
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    b /= a.ncb;  // a single block of 16 input channels
    const int mb = int(b % a.nmb);
    const int64_t split = b / a.nmb;
    const int64_t br0 = split * a.nbricks / a.nsplit, br1 = (split + 1) * a.nbricks / a.nsplit;
    const int kd0 = tg;
    const int co0 = mb * 64;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    const int nxv = a.biz * a.biy * rp;
    const int nxi = dl_round(nxv * 2) / kThreads, ndi = dl_round(bov * 8) / kThreads;

    // the thread's load units, brick invariant. Input: unit s = 16-byte half
    // s & 1 (channels 8 (s & 1) ..) of voxel slot s >> 1; packed
    // z << 20 | y << 10 | x << 1 | half, -1 past the row or brick. dy: unit s =
    // 16-byte unit p = s & 7 of voxel f = s >> 3, holding channels 8 q .., q =
    // p ^ 4 ((f / 2) % 2); packed oz << 22 | oy << 12 | ox << 3 | q.
    int px[kTrXU], pd[kTrDU];
#pragma unroll
    for (int i = 0; i < kTrXU; ++i) {
        const int sl = tid + i * kThreads;
        const int v = sl >> 1, h = sl & 1;
        const int x = v % rp, r = v / rp;
        px[i] = (v < nxv && x < a.bix) ? (((r / a.biy) << 20) | ((r % a.biy) << 10) | (x << 1) | h) : -1;
    }
#pragma unroll
    for (int i = 0; i < kTrDU; ++i) {
        const int sl = tid + i * kThreads;
        const int f = sl >> 3, q = (sl & 7) ^ (((f >> 1) & 1) << 2);
        const int ox = f % a.BO[2], oy = (f / a.BO[2]) % a.BO[1], oz = f / (a.BO[2] * a.BO[1]);
        pd[i] = f < bov ? ((oz << 22) | (oy << 12) | (ox << 3) | q) : -1;
    }
    const int P0 = int(a.P[0]), P1 = int(a.P[1]), P2 = int(a.P[2]);
    const int O0 = int(a.O[0]), O1 = int(a.O[1]), O2 = int(a.O[2]);
    const int cout = int(a.cout);
    constexpr uint32_t kOut = 0xFFFFFFF0u;
    // per axis: first tile row with data and the count of such rows (all P
    // rows; with a folded halo, a margin without a slab is zero, not read)
    int V[6] = {0, P0, 0, P1, 0, P2};
    if constexpr (FOLD) {
        for (int k = 0; k < 3; ++k) {
            if (!((a.fold.mask >> k) & 1u)) continue;
            const int lo = a.fold.slab[k][0] ? 0 : int(a.fold.lo[k]);
            const int hi = a.fold.slab[k][1] ? int(a.P[k]) : int(a.fold.lo[k] + a.fold.ext[k]);
            V[2 * k] = lo;
            V[2 * k + 1] = hi - lo;
        }
    }

    // loads of brick br into the buffer at byte offset boff
    auto stage = [&](int64_t br, int boff) {
        int64_t nn, ob[3];
        brick_origin(a, br, nn, ob);
        const int i0 = int(ob[0]) * a.S[0] + kd0 - a.pad[0], i1 = int(ob[1]) * a.S[1] - a.pad[1],
                  i2 = int(ob[2]) - a.pad[2];
        const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.tile) + int64_t(nn) * xbatch, short(0), int(xbatch), 0x00020000);
        const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.dy) + int64_t(nn) * dbatch, short(0), int(dbatch), 0x00020000);
        // with a folded halo, a brick whose input rows touch a margin takes each
        // voxel from its own buffer (tile or slab, per lane: global->LDS loads
        // with per-lane addresses, zero padding from a zeroed source); every
        // other brick reads the tile as without one
        bool plain = true;
        if constexpr (FOLD) {
            const int64_t fi[3] = {i0, i1, i2}, fe[3] = {a.biz, a.biy, a.bix};
            for (int k = 0; k < 3; ++k)
                if ((a.fold.mask >> k) & 1u)
                    plain = plain && (fi[k] >= a.fold.lo[k] || !a.fold.slab[k][0]) &&
                            (fi[k] + fe[k] <= a.fold.lo[k] + a.fold.ext[k] || !a.fold.slab[k][1]);
        }
        if (plain) {
#pragma unroll
            for (int i = 0; i < kTrXU; ++i) {
                if (i < nxi) {
                    const int c = px[i];
                    const int t0 = i0 + (c >> 20), t1 = i1 + ((c >> 10) & 1023), t2 = i2 + ((c >> 1) & 511);
                    // in range of the tile's rows that hold data (margins without a
                    // slab are zero)
                    const bool ok = c >= 0 && uint32_t(t0 - V[0]) < uint32_t(V[1]) &&
                                    uint32_t(t1 - V[2]) < uint32_t(V[3]) && uint32_t(t2 - V[4]) < uint32_t(V[5]);
                    const uint32_t off = ((uint32_t(t0 * P1 + t1) * uint32_t(P2) + uint32_t(t2)) * 16u +
                                          uint32_t(8 * (c & 1))) * 2u;
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, SC_LDSW(lds + boff + i * 4096 + wave * 1024), 16,
                                                             ok ? off : kOut, 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < kTrXU; ++i) {
                if (i < nxi) {
                    const int c = px[i];
                    const int t0 = i0 + (c >> 20), t1 = i1 + ((c >> 10) & 1023), t2 = i2 + ((c >> 1) & 511);
                    const bool ok = c >= 0 && uint32_t(t0) < uint32_t(P0) && uint32_t(t1) < uint32_t(P1) &&
                                    uint32_t(t2) < uint32_t(P2);
                    const char* src = a.zeros;
                    if (ok) {
                        const char* v = fold_voxel(a.fold, a.tile, nn, t0, t1, t2, 32);
                        if (v) src = v + 16 * (c & 1);
                    }
                    __builtin_amdgcn_global_load_lds(src, SC_LDSW(lds + boff + i * 4096 + wave * 1024), 16, 0, 0);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kTrDU; ++i) {
            if (i < ndi) {
                const int c = pd[i];
                const int o0 = int(ob[0]) + (c >> 22), o1 = int(ob[1]) + ((c >> 12) & 1023),
                          o2 = int(ob[2]) + ((c >> 3) & 511);
                const bool ok = c >= 0 && o0 < O0 && o1 < O1 && o2 < O2;
                const uint32_t off = ((uint32_t(o0 * O1 + o1) * uint32_t(O2) + uint32_t(o2)) * uint32_t(cout) +
                                      uint32_t(co0 + 8 * (c & 7))) * 2u;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rd, SC_LDSW(lds + boff + dy_off + i * 4096 + wave * 1024), 16, ok ? off : kOut, 0, 0, 0);
            }
        }
    };

    f32x16_w acc[NT > 0 ? NT : 1];  // a 1x1 kernel leaves waves 2, 3 without tiles
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;

    const uint32_t lds0 = lds_addr(lds);
    const uint32_t colb = uint32_t((li & 3) * 8);
    // per-lane read offsets within a buffer. A: voxel 8 gk + vr (+ 4) of the K
    // step, chunk 2 ch + gh; run p: row 2 p + gh; W run: row K1 - 1, one voxel
    // further on for gh = 1
    const uint32_t cA = uint32_t(dy_off) + uint32_t((8 * gk + vr) * 128) +
                        uint32_t(((2 * ch + gh) ^ (((vr >> 1) & 1) << 1)) * 32) + colb;
    uint32_t cX[TL::NRUN];
#pragma unroll
    for (int r = 0; r < TL::NRUN; ++r)
        cX[r] = r < TL::NR ? uint32_t(((2 * r + gh) * rp + 8 * gk + vr) * 32) + colb
                           : uint32_t(((K1 - 1) * rp + 8 * gk + gh + vr) * 32) + colb;
    const int nks = bov / 16;

    // operand reads of K step ks (voxels 16 ks .. of the brick, at (oz, oy, ox)):
    // a tile's window w .. w + 7 is two reads at voxel offsets w and w + 4 of its
    // run, straight into the product's operand registers
    auto issue = [&](PrOps<NT>& o, uint32_t aA, uint32_t U) {
        o.a[0] = lds_read_tr16_b64(aA);
        o.a[1] = lds_read_tr16_b64<512>(aA);
        uint32_t ad[TL::NRUN];
#pragma unroll
        for (int r = 0; r < TL::NRUN; ++r)
            if (TL::uses(TH, r)) ad[r] = U + cX[r];
        static_for<NT>([&](auto ic) {
            constexpr int t = T0 + decltype(ic)::value;
            o.b[decltype(ic)::value][0] = lds_read_tr16_b64<32 * TL::win(t)>(ad[TL::run(t)]);
            o.b[decltype(ic)::value][1] = lds_read_tr16_b64<32 * TL::win(t) + 128>(ad[TL::run(t)]);
        });
    };
    auto compute = [&](PrOps<NT>& o) {
        uint2 a0 = o.a[0], a1 = o.a[1];
        lds_ready(a0);
        lds_ready(a1);
        const uint4 av = make_uint4(a0.x, a0.y, a1.x, a1.y);
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            uint2 b0 = o.b[i][0], b1 = o.b[i][1];
            lds_ready(b0);
            lds_ready(b1);
            const uint4 bv = make_uint4(b0.x, b0.y, b1.x, b1.y);
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                              __builtin_bit_cast(bf16x8_w, bv), acc[i], 0, 0, 0);
        }
    };

    if (br0 < br1) stage(br0, 0);
    for (int64_t br = br0; br < br1; ++br) {
        const int cur = int((br - br0) & 1);
        // this thread's loads of brick br have landed; after the barrier every
        // thread's have, and every wave is done with the other buffer
        wait_vm_barrier<0>();
        if (br + 1 < br1) stage(br + 1, (cur ^ 1) * bufb);
        if constexpr (NT > 0) {
            // step positions advance by 16 voxels along W, then by a row, then
            // by a plane of the brick: byte offsets of the run starts (U) and
            // of dy (aA) move by wave-uniform increments
            const uint32_t base = lds0 + uint32_t(cur * bufb);
            const uint32_t rowstep = uint32_t((rp - a.BO[2]) * 32);
            const uint32_t planestep = uint32_t((a.biy - a.BO[1]) * rp * 32);
            uint32_t aA = base + cA, U = base;
            int ox = 0, oy = 0;
            auto advance = [&]() {
                aA += 2048u;
                U += 512u;
                ox += 16;
                if (ox == a.BO[2]) {
                    ox = 0;
                    U += rowstep;
                    if (++oy == a.BO[1]) {
                        oy = 0;
                        U += planestep;
                    }
                }
            };
            PrOps<NT> o0, o1;
            issue(o0, aA, U);
            for (int ks = 0; ks < nks; ks += 2) {  // nks is even
                advance();
                lds_wait<0>();
                issue(o1, aA, U);
                compute(o0);
                // the last pair re-reads its second step: same registers every
                // iteration, no step past the brick
                if (ks + 2 < nks) advance();
                lds_wait<0>();
                issue(o0, aA, U);
                compute(o1);
            }
        }
    }
    lds_wait<0>();  // the last re-read has landed
    // accumulator element e of lane l: output channel 32 ch + 8 (e / 4) +
    // 4 (l / 32) + e % 4, column l % 32 = 16 gh + ci; stored in the layout
    // [16-channel group][tap][16 (co % 16 / 4) + ci][co % 4]
    float* out = a.part + ((((split * a.nmb + mb) * a.ncb) * a.ntg + tg) * int64_t(a.blk));
#pragma unroll
    for (int i = 0; i < NT; ++i) {
        const int t = T0 + i;
        const int kh = gh ? TL::kh(t, 1) : TL::kh(t, 0), kw = gh ? TL::kw(t, 1) : TL::kw(t, 0);
        if (kh >= K1 || kw >= K2) continue;
        const int ti = kh * K2 + kw;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int co = 32 * ch + 8 * (e >> 2) + 4 * gk + (e & 3);
            out[(((co >> 4) * TG + ti) * 64 + 16 * ((co & 15) >> 2) + li) * 4 + (co & 3)] = acc[i][e];
        }
    }
}

template <int K1, int K2, bool FOLD>
__global__ __launch_bounds__(kThreads, 2) void wgrad_bf16_pr(WgArgs a, int rp, int dy_off, int bufb, uint32_t xbatch,
                                                             uint32_t dbatch)
{
    // waves 0, 1 and waves 2, 3 (a wave-uniform choice, made scalar so that the
    // compiler keeps the step's bookkeeping in scalar registers)
    if (__builtin_amdgcn_readfirstlane(threadIdx.x >> 7) == 0)
        wgrad_bf16_pr_body<K1, K2, 0, FOLD>(a, rp, dy_off, bufb, xbatch, dbatch);
    else
        wgrad_bf16_pr_body<K1, K2, 1, FOLD>(a, rp, dy_off, bufb, xbatch, dbatch);
}

template <int TPW>
__global__ __launch_bounds__(kThreads, 2) void wgrad_f32_tiled(WgArgs a)
{
    extern __shared__ uint4 lds4[];
    float* xs = reinterpret_cast<float*>(lds4);
    float* ds = reinterpret_cast<float*>(reinterpret_cast<char*>(lds4) + a.dy_off);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 5;
    const int l32 = lane & 31;

    int64_t b = xcd_remap(blockIdx.x, a.nblocks);
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    const int cb = int(b % a.ncb);
    b /= a.ncb;
    const int mb = int(b % a.nmb);
    const int64_t split = b / a.nmb;
    const int64_t br0 = split * a.nbricks / a.nsplit, br1 = (split + 1) * a.nbricks / a.nsplit;
    const int64_t co0 = int64_t(mb) * 32, ci0 = int64_t(cb) * 32;
    const int taps = a.K[0] * a.K[1] * a.K[2];
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    const int biv = a.biz * a.biy * a.bix;
    const float* tile = reinterpret_cast<const float*>(a.tile);
    const float* dy = reinterpret_cast<const float*>(a.dy);
    const bool xvec = a.xvec != 0, dvec = a.dvec != 0;

    // this wave's taps: t = tg * kdg + wave + 4 i
    int toff[TPW];
    bool tok[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tl = wave + 4 * i;
        const int t = tg * a.kdg + tl;
        tok[i] = tl < a.kdg && t < taps;
        const int tt = tok[i] ? t : 0;
        const int kw = tt % a.K[2], kh = (tt / a.K[2]) % a.K[1], kd = tt / (a.K[2] * a.K[1]);
        toff[i] = (kd * a.biy + kh) * a.bix + kw;
    }
    f32x16_w acc[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;

    for (int64_t br = br0; br < br1; ++br) {
        int64_t nn, ob[3];
        brick_origin(a, br, nn, ob);
        const int64_t i0 = ob[0] * a.S[0] - a.pad[0];
        const int64_t i1 = ob[1] * a.S[1] - a.pad[1];
        const int64_t i2 = ob[2] * a.S[2] - a.pad[2];
        __syncthreads();
        // staging: a thread keeps its (x, 4-channel unit) column and steps over
        // rows (one division per row) when a row of units fits the block
        auto stage_x = [&](int q, int x, int row) {
            const int y = row % a.biy;
            const int z = row / a.biy;
            const int64_t t0 = i0 + z, t1 = i1 + y, t2 = i2 + x;
            const int64_t c = ci0 + 4 * q;
            float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
            const float* vox = nullptr;
            if (t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] && c < a.cin)
                vox = a.fold.mask
                          ? reinterpret_cast<const float*>(fold_voxel(a.fold, a.tile, nn, t0, t1, t2, a.cin * 4))
                          : tile + (((nn * a.P[0] + t0) * a.P[1] + t1) * a.P[2] + t2) * a.cin;
            if (vox) {
                const float* src = vox + c;
                if (xvec && c + 4 <= a.cin) {
                    val = *reinterpret_cast<const float4*>(src);
                } else {
                    float tmp[4];
                    for (int e = 0; e < 4; ++e) tmp[e] = (c + e < a.cin) ? src[e] : 0.f;
                    val = make_float4(tmp[0], tmp[1], tmp[2], tmp[3]);
                }
            }
            reinterpret_cast<float4*>(xs)[(row * a.bix + x) * 8 + q] = val;
        };
        {
            const int rowlen = a.bix * 8, rows = a.biz * a.biy;
            if (rowlen <= kThreads) {
                const int rpp = kThreads / rowlen;
                const int r0 = int(threadIdx.x) / rowlen, cu = int(threadIdx.x) - r0 * rowlen;
                if (r0 < rpp)
                    for (int row = r0; row < rows; row += rpp) stage_x(cu % 8, cu / 8, row);
            } else {
                for (int u = threadIdx.x; u < biv * 8; u += kThreads) {
                    const int v = u / 8;
                    stage_x(u % 8, v % a.bix, v / a.bix);
                }
            }
        }
        const int bove = bov + (bov & 1);
        auto stage_dy = [&](int q, int f) {
            const int ox = f % a.BO[2];
            const int oy = (f / a.BO[2]) % a.BO[1];
            const int oz = f / (a.BO[2] * a.BO[1]);
            const int64_t o0 = ob[0] + oz, o1 = ob[1] + oy, o2 = ob[2] + ox;
            const int64_t c = co0 + 4 * q;
            float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
            if (f < bov && o0 < a.O[0] && o1 < a.O[1] && o2 < a.O[2] && c < a.cout) {
                const float* src = dy + (((nn * a.O[0] + o0) * a.O[1] + o1) * a.O[2] + o2) * a.cout + c;
                if (dvec && c + 4 <= a.cout) {
                    val = *reinterpret_cast<const float4*>(src);
                } else {
                    float tmp[4];
                    for (int e = 0; e < 4; ++e) tmp[e] = (c + e < a.cout) ? src[e] : 0.f;
                    val = make_float4(tmp[0], tmp[1], tmp[2], tmp[3]);
                }
            }
            reinterpret_cast<float4*>(ds)[f * 8 + q] = val;
        };
        for (int u = threadIdx.x; u < bove * 8; u += kThreads) stage_dy(u % 8, u / 8);
        __syncthreads();
        // output voxel f = 2 ks + g of the brick; its coordinates advance by
        // carries (a lane past the brick's end uses voxel 0: its dy row is zero)
        int ox = g % a.BO[2], oy = (g / a.BO[2]) % a.BO[1], oz = g / (a.BO[2] * a.BO[1]);
        for (int ks = 0; ks < bove / 2; ++ks) {
            const int f = 2 * ks + g;
            if (ks > 0) {
                ox += 2;
                while (ox >= a.BO[2]) {
                    ox -= a.BO[2];
                    if (++oy == a.BO[1]) {
                        oy = 0;
                        ++oz;
                    }
                }
            }
            const bool live = f < bov;
            const int vin =
                live ? (oz * a.S[0] * a.biy + oy * a.S[1]) * a.bix + ox * a.S[2] : 0;
            const float av = ds[f * 32 + l32];
#pragma unroll
            for (int i = 0; i < TPW; ++i) {
                if (!tok[i]) continue;
                const float bv = xs[(vin + toff[i]) * 32 + l32];
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[i], 0, 0, 0);
            }
        }
    }
    float4* out = reinterpret_cast<float4*>(a.part + (((split * a.nmb + mb) * a.ncb + cb) * a.ntg + tg) * int64_t(a.blk) +
                                            int64_t(wave) * TPW * 1024);
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            out[(i * 64 + lane) * 4 + r4] =
                make_float4(acc[i][4 * r4], acc[i][4 * r4 + 1], acc[i][4 * r4 + 2], acc[i][4 * r4 + 3]);
}

// fp32 with direct global->LDS loads: the staging of a brick is one 16-byte
// buffer load per thread and 4 KiB of LDS (unit u = thread + 256 i is float4 u
// of the input copy: voxel u / 8, channels 4 (u % 8) ..), written by the load
// itself with no register copy and no LDS store instruction; an offset past
// the buffer (a voxel outside the tile, a unit past the brick) loads zeros.
// Each thread's unit coordinates inside a brick are the same for every brick,
// so they are packed into registers once. The K steps run as a software
// pipeline (the operands of step ks + 1 are read while the MFMAs of step ks
// run, every tap slot multiplies, no branch). Two workgroups per compute unit
// alternate between loading and multiplying. Same bricks, K steps and taps as
// wgrad_f32_tiled, in the same order: the partials are bit-identical.
constexpr int kDlXU = 20;    // input load instructions per thread (80 KiB)
constexpr int kDlDU = 3;     // dy load instructions per thread (bricks of <= 64 outputs)
constexpr int kDlTab = 66;   // entries of the per-voxel input offset table

struct DlLayout {
    int dy_off, tab_off, bytes;
};

inline DlLayout dl_layout(const WgArgs& a)
{
    const int biv = a.biz * a.biy * a.bix;
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    DlLayout L;
    L.dy_off = dl_round(biv * 8) * 16;
    L.tab_off = L.dy_off + dl_round((bov + (bov & 1)) * 8) * 16;
    L.bytes = L.tab_off + kDlTab * 4;
    return L;
}

// FOLD: the halo along axis 0 folded into the loads (the only axis with
// margins): padded planes below fold.lo[0] come from the lo slab, planes from
// fold.lo[0] + fold.ext[0] on from the hi slab (plane strides as in the tile; a
// missing slab is a zero-length buffer, so its planes load as zeros). A lane
// picks its buffer per unit; the load of each buffer goes out under the exec
// mask of its lanes.
template <int TPW, bool FOLD>
__global__ __launch_bounds__(kThreads, 2) void wgrad_f32_dl(WgArgs a, int dy_off, int tab_off, uint32_t xbatch,
                                                            uint32_t dbatch, uint32_t fbatch_lo, uint32_t fbatch_hi)
{
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const float* xs = reinterpret_cast<const float*>(lds);
    const float* ds = reinterpret_cast<const float*>(lds + dy_off);
    int* vtab = reinterpret_cast<int*>(lds + tab_off);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int g = lane >> 5;
    const int l32 = lane & 31;

    int64_t b = xcd_remap(blockIdx.x, a.nblocks);
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    const int cb = int(b % a.ncb);
    b /= a.ncb;
    const int mb = int(b % a.nmb);
    const int64_t split = b / a.nmb;
    const int64_t br0 = split * a.nbricks / a.nsplit, br1 = (split + 1) * a.nbricks / a.nsplit;
    const int co0 = mb * 32, ci0 = cb * 32;
    const int taps = a.K[0] * a.K[1] * a.K[2];
    const int bov = a.BO[0] * a.BO[1] * a.BO[2];
    const int bove = bov + (bov & 1);
    const int biv = a.biz * a.biy * a.bix;
    const int nxi = dl_round(biv * 8) / kThreads, ndi = dl_round(bove * 8) / kThreads;

    // tap slots past the last tap multiply tap 0's operands (no branch in the
    // MFMA sequence); the reduction never reads their partials
    int toff[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tl = wave + 4 * i;
        const int t = tg * a.kdg + tl;
        const int tt = (tl < a.kdg && t < taps) ? t : 0;
        const int kw = tt % a.K[2], kh = (tt / a.K[2]) % a.K[1], kd = tt / (a.K[2] * a.K[1]);
        toff[i] = ((kd * a.biy + kh) * a.bix + kw) * 32 + l32;
    }
    f32x16_w acc[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;

    // the thread's units: voxel (z, y, x) of the input brick packed as
    // z << 20 | y << 10 | x, output voxel (oz, oy, ox) of the dy brick likewise;
    // -1 for a unit past the brick
    const int q = tid & 7;
    int px[kDlXU], pd[kDlDU];
#pragma unroll
    for (int i = 0; i < kDlXU; ++i) {
        const int v = (tid + i * kThreads) >> 3;
        const int x = v % a.bix, r = v / a.bix;
        px[i] = v < biv ? (((r / a.biy) << 20) | ((r % a.biy) << 10) | x) : -1;
    }
#pragma unroll
    for (int i = 0; i < kDlDU; ++i) {
        const int f = (tid + i * kThreads) >> 3;
        const int ox = f % a.BO[2], oy = (f / a.BO[2]) % a.BO[1], oz = f / (a.BO[2] * a.BO[1]);
        pd[i] = f < bov ? ((oz << 20) | (oy << 10) | ox) : -1;
    }
    for (int f = tid; f < bove; f += kThreads) {
        const int ox = f % a.BO[2], oy = (f / a.BO[2]) % a.BO[1], oz = f / (a.BO[2] * a.BO[1]);
        vtab[f] = f < bov ? ((oz * a.S[0] * a.biy + oy * a.S[1]) * a.bix + ox * a.S[2]) * 32 : 0;
    }
    const int P0 = int(a.P[0]), P1 = int(a.P[1]), P2 = int(a.P[2]);
    const int O0 = int(a.O[0]), O1 = int(a.O[1]), O2 = int(a.O[2]);
    const int cin = int(a.cin), cout = int(a.cout);
    const bool cok = ci0 + 4 * q < cin, dok = co0 + 4 * q < cout;
    constexpr uint32_t kOut = 0xFFFFFFF0u;  // past every buffer: loads zeros

    for (int64_t br = br0; br < br1; ++br) {
        int64_t nn, ob[3];
        brick_origin(a, br, nn, ob);
        const int i0 = int(ob[0] * a.S[0] - a.pad[0]), i1 = int(ob[1] * a.S[1] - a.pad[1]),
                  i2 = int(ob[2] * a.S[2] - a.pad[2]);
        __syncthreads();  // every wave is done reading the previous brick
        const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.tile) + int64_t(nn) * xbatch, short(0), int(xbatch), 0x00020000);
        const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.dy) + int64_t(nn) * dbatch, short(0), int(dbatch), 0x00020000);
        __amdgpu_buffer_rsrc_t rl = rx, rh = rx;
        if (FOLD) {
            const char* sl = a.fold.slab[0][0];
            const char* sh = a.fold.slab[0][1];
            rl = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(sl ? sl + int64_t(nn) * fbatch_lo : a.tile),
                                                   short(0), sl ? int(fbatch_lo) : 0, 0x00020000);
            rh = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(sh ? sh + int64_t(nn) * fbatch_hi : a.tile),
                                                   short(0), sh ? int(fbatch_hi) : 0, 0x00020000);
        }
        const int flo = FOLD ? int(a.fold.lo[0]) : 0, fhi = FOLD ? int(a.fold.lo[0] + a.fold.ext[0]) : P0;
#pragma unroll
        for (int i = 0; i < kDlXU; ++i) {
            if (i < nxi) {
                const int c = px[i];
                const int t0 = i0 + (c >> 20), t1 = i1 + ((c >> 10) & 1023), t2 = i2 + (c & 1023);
                const bool ok = c >= 0 && cok && uint32_t(t0) < uint32_t(P0) && uint32_t(t1) < uint32_t(P1) &&
                                uint32_t(t2) < uint32_t(P2);
                const uint32_t off = ((uint32_t(t0 * P1 + t1) * uint32_t(P2) + uint32_t(t2)) * uint32_t(cin) +
                                      uint32_t(ci0 + 4 * q)) * 4u;
                char* dst = lds + i * 4096 + wave * 1024;
                if (FOLD && t0 < flo) {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, SC_LDSW(dst), 16, ok ? off : kOut, 0, 0, 0);
                } else if (FOLD && t0 >= fhi) {
                    const uint32_t o = off - uint32_t(fhi) * uint32_t(P1) * uint32_t(P2) * uint32_t(cin) * 4u;
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, SC_LDSW(dst), 16, ok ? o : kOut, 0, 0, 0);
                } else {
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, SC_LDSW(dst), 16, ok ? off : kOut, 0, 0, 0);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kDlDU; ++i) {
            if (i < ndi) {
                const int c = pd[i];
                const int o0 = int(ob[0]) + (c >> 20), o1 = int(ob[1]) + ((c >> 10) & 1023),
                          o2 = int(ob[2]) + (c & 1023);
                const bool ok = c >= 0 && dok && o0 < O0 && o1 < O1 && o2 < O2;
                const uint32_t off = ((uint32_t(o0 * O1 + o1) * uint32_t(O2) + uint32_t(o2)) * uint32_t(cout) +
                                      uint32_t(co0 + 4 * q)) * 4u;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, SC_LDSW(lds + dy_off + i * 4096 + wave * 1024), 16,
                                                         ok ? off : kOut, 0, 0, 0);
            }
        }
        wait_vm_barrier<0>();  // the brick's loads have landed, for every wave
        // software pipeline over the K steps: the operands of step ks + 1 and the
        // input offset of step ks + 2 are read while the MFMAs of step ks run
        const int nks = bove / 2;
        float av = ds[g * 32 + l32];
        float bv[TPW];
        {
            const int v0 = vtab[g];
#pragma unroll
            for (int i = 0; i < TPW; ++i) bv[i] = xs[v0 + toff[i]];
        }
        int vin1 = nks > 1 ? vtab[2 + g] : 0;
        for (int ks = 0; ks < nks; ++ks) {
            float avn = 0.f, bvn[TPW];
            int vin2 = 0;
            if (ks + 1 < nks) {
                avn = ds[(2 * ks + 2 + g) * 32 + l32];
#pragma unroll
                for (int i = 0; i < TPW; ++i) bvn[i] = xs[vin1 + toff[i]];
                if (ks + 2 < nks) vin2 = vtab[2 * ks + 4 + g];
            }
#pragma unroll
            for (int i = 0; i < TPW; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv[i], acc[i], 0, 0, 0);
            av = avn;
#pragma unroll
            for (int i = 0; i < TPW; ++i) bv[i] = bvn[i];
            vin1 = vin2;
        }
    }
    float4* out = reinterpret_cast<float4*>(a.part + (((split * a.nmb + mb) * a.ncb + cb) * a.ntg + tg) * int64_t(a.blk) +
                                            int64_t(wave) * TPW * 1024);
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            out[(i * 64 + lane) * 4 + r4] =
                make_float4(acc[i][4 * r4], acc[i][4 * r4 + 1], acc[i][4 * r4 + 2], acc[i][4 * r4 + 3]);
}

// Sum the split partials in split order and scatter into dw[co][ci][tap].
// One thread per partial float of one (mb, cb, tg) block: reads are coalesced.
__global__ __launch_bounds__(256) void wgrad_reduce(WgArgs a, int kind, int kdg, int k1, int k2, int wco)
{
    const int64_t groups = int64_t(a.nmb) * a.ncb * a.ntg;
    const int64_t total = groups * a.blk;
    const int taps = a.K[0] * a.K[1] * a.K[2];
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        const int64_t grp = e / a.blk;
        const int p = int(e % a.blk);
        const int tg = int(grp % a.ntg);
        const int cb = int((grp / a.ntg) % a.ncb);
        const int mb = int(grp / (int64_t(a.ntg) * a.ncb));
        int64_t co, ci;
        int tap;
        if (kind == 1) {
            const int wci_n = 4 / wco;
            const int tgs = kdg * k1 * k2;
            const int r = p % 4, lane = (p / 4) % 64, ti = (p / 256) % tgs, wave = p / (256 * tgs);
            const int wc = wave / wci_n, wi = wave % wci_n;
            co = int64_t(mb) * wco * 16 + wc * 16 + 4 * (lane / 16) + r;
            ci = int64_t(cb) * wci_n * 16 + wi * 16 + (lane % 16);
            const int kw = ti % k2, kh = (ti / k2) % k1, kdl = ti / (k2 * k1);
            tap = ((tg * kdg + kdl) * a.K[1] + kh) * a.K[2] + kw;
        } else {
            const int tpw = a.blk / (4 * 1024);
            const int r = p % 16, lane = (p / 16) % 64, i = (p / 1024) % tpw, wave = p / (1024 * tpw);
            const int row = 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
            co = int64_t(mb) * 32 + row;
            ci = int64_t(cb) * 32 + (lane % 32);
            const int tl = wave + 4 * i;
            tap = tg * kdg + tl;
            if (tl >= kdg) continue;
        }
        if (co >= a.cout || ci >= a.cin || tap >= taps) continue;
        // eight interleaved partial sums (split index mod 8), combined in a fixed
        // tree: a fixed summation order with eight loads in flight
        float s8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        int64_t sp = 0;
        for (; sp + 8 <= a.nsplit; sp += 8) {
#pragma unroll
            for (int j = 0; j < 8; ++j) s8[j] += a.part[(sp + j) * total + e];
        }
        for (int j = 0; sp + j < a.nsplit; ++j) s8[j] += a.part[(sp + j) * total + e];
        const float s = ((s8[0] + s8[1]) + (s8[2] + s8[3])) + ((s8[4] + s8[5]) + (s8[6] + s8[7]));
        a.dw[(co * a.cin + ci) * taps + tap] = s;
    }
}

bool bf16_instance(int kdg, int k1, int k2)
{
    return (kdg == 3 && k1 == 3 && k2 == 3) || (kdg == 1 && k1 == 3 && k2 == 3) || (kdg == 1 && k1 == 5 && k2 == 5) ||
           (kdg == 1 && k1 == 1 && (k2 == 1 || k2 == 3 || k2 == 5));
}

PlanW plan_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    PlanW pl{};
    pl.kind = 0;
    if (force_generic()) return pl;
    const int64_t taps = cv.taps();
    for (int k = 0; k < 3; ++k)
        if (cv.K[k] > 64 || cv.S[k] > 64 || cv.O[k] > (int64_t(1) << 30) || std::abs(cv.pad[k]) > (1 << 29)) return pl;
    if (t.c > 4096 || cv.cout > 4096) return pl;
    WgArgs a{};
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
    const size_t kLds = 80 * 1024;
    if (dt == SHARD_BF16) {
        if (cv.S[2] != 1 || cv.K[2] > 8) return pl;
        int kdg = (cv.K[0] * cv.K[1] * cv.K[2] <= 27) ? int(cv.K[0]) : 1;
        if (!bf16_instance(kdg, int(cv.K[1]), int(cv.K[2]))) return pl;
        const int wco = t.c <= 16 ? 4 : 2, wci = 4 / wco;
        const int nco = wco * 16, nci = wci * 16;
        // the row-pair kernel's brick (when its shape applies): W extent a
        // multiple of 16 (a K step is one W run), double-buffered staging within
        // two workgroups' LDS per CU
        double best = 1e300;
        const bool pr_shape = kdg == 1 && t.c == 16 && cv.cout % 64 == 0 && cv.K[2] <= 5 && cv.S[0] == 1 &&
                              cv.S[1] == 1 && cv.S[2] == 1 && !force_tiled();
        for (int b2 : {16, 32, 64}) {
            for (int b1 = 1; b1 <= 64 && pr_shape; b1 *= 2) {
                for (int b0 = 1; b0 <= 64; b0 *= 2) {
                    const int bov = b0 * b1 * b2;
                    if (bov % 32 != 0 || bov > kTrDU * kThreads / 8) continue;
                    if ((b0 > 1 && b0 > cv.O[0]) || (b1 > 1 && b1 > cv.O[1])) continue;
                    WgArgs c{};
                    c.BO[0] = b0;
                    c.BO[1] = b1;
                    c.BO[2] = b2;
                    c.biz = b0;
                    c.biy = int(b1 - 1 + cv.K[1]);
                    c.bix = int(b2 + cv.K[2] - 1);
                    const PrLayout L = pr_layout(c);
                    if (c.biz * c.biy * L.rp * 2 > kTrXU * kThreads || L.bytes > int(kLds)) continue;
                    const int bixp = b2 + 8;
                    const int cs = int(round_up(c.biz * c.biy * bixp, 16) + 8), csd = int(round_up(bov, 16) + 8);
                    const int dy_off = int(round_up(int64_t(nci) * cs * 2, 16));
                    const size_t lds = size_t(dy_off) + size_t(nco) * csd * 2;  // the tiled kernels' need
                    if (lds > kLds) continue;
                    double eff = 1.0;
                    const int64_t bo[3] = {b0, b1, b2};
                    for (int k = 0; k < 3; ++k) eff *= double(cv.O[k]) / double(ceil_div(cv.O[k], bo[k]) * bo[k]);
                    const double cost = double(c.biz * c.biy * L.rp * 32 + bov * 128) / bov / eff + 8192.0 / bov;
                    if (cost < best) {
                        best = cost;
                        a.BO[0] = b0;
                        a.BO[1] = b1;
                        a.BO[2] = b2;
                        a.biz = c.biz;
                        a.biy = c.biy;
                        a.bix = c.bix;
                        a.bixp = bixp;
                        a.cs = cs;
                        a.csd = csd;
                        a.dy_off = dy_off;
                        pl.lds = lds;
                    }
                }
            }
        }
        // otherwise: W extent a multiple of 8 (an 8-voxel K group stays in one row)
        for (int b2 : {32, 64, 16, 8}) {
            if (best < 1e299) break;
            for (int b1 = 1; b1 <= 64; b1 *= 2) {
                for (int b0 = 1; b0 <= 64; b0 *= 2) {
                    const int bov = b0 * b1 * b2;
                    if (bov % 32 != 0 || bov > 1024) continue;
                    if (b0 > 1 && b0 > cv.O[0]) continue;
                    if (b1 > 1 && b1 > cv.O[1]) continue;
                    const int biz = int((b0 - 1) * cv.S[0] + kdg);
                    const int biy = int((b1 - 1) * cv.S[1] + cv.K[1]);
                    const int bix = int(b2 + cv.K[2] - 1);
                    const int bixp = b2 + 8;
                    int cs = biz * biy * bixp;
                    cs = int(round_up(cs, 16) + 8);
                    const int csd = int(round_up(bov, 16) + 8);
                    const int dy_off = int(round_up(int64_t(nci) * cs * 2, 16));
                    const size_t lds = size_t(dy_off) + size_t(nco) * csd * 2;
                    if (lds > kLds) continue;
                    double eff = 1.0;
                    const int64_t bo[3] = {b0, b1, b2};
                    for (int k = 0; k < 3; ++k) eff *= double(cv.O[k]) / double(ceil_div(cv.O[k], bo[k]) * bo[k]);
                    const double cost = (double(biz * biy * bix) * nci / bov + double(nco)) / eff +
                                        4096.0 / bov;  // staging bytes per output voxel, plus a per-brick overhead
                    if (cost < best) {
                        best = cost;
                        a.BO[0] = b0;
                        a.BO[1] = b1;
                        a.BO[2] = b2;
                        a.biz = biz;
                        a.biy = biy;
                        a.bix = bix;
                        a.bixp = bixp;
                        a.cs = cs;
                        a.csd = csd;
                        a.dy_off = dy_off;
                        pl.lds = lds;
                    }
                }
            }
        }
        if (best >= 1e299) return pl;
        a.kdg = kdg;
        a.nmb = int32_t(ceil_div(cv.cout, nco));
        a.ncb = int32_t(ceil_div(t.c, nci));
        a.ntg = int32_t(cv.K[0] / kdg);
        a.blk = 4 * kdg * int(cv.K[1] * cv.K[2]) * 256;
        a.wco = wco;
        a.wci = wci;
        pl.kind = 1;
        pl.kdg = kdg;
        pl.k1 = int(cv.K[1]);
        pl.k2 = int(cv.K[2]);
        pl.wco = wco;
    } else {
        const int tpw = 7;
        const int tgs = 4 * tpw;
        // brick: any shape with <= 64 outputs whose input footprint fits
        double best = 1e300;
        for (int b2 = 1; b2 <= 64; b2 *= 2)
            for (int b1 = 1; b1 <= 64; b1 *= 2)
                for (int b0 = 1; b0 <= 64; b0 *= 2) {
                    const int bov = b0 * b1 * b2;
                    if (bov > 64 || bov < 2) continue;
                    if ((b0 > 1 && b0 > cv.O[0]) || (b1 > 1 && b1 > cv.O[1]) || (b2 > 1 && b2 > cv.O[2])) continue;
                    const int biz = int((b0 - 1) * cv.S[0] + cv.K[0]);
                    const int biy = int((b1 - 1) * cv.S[1] + cv.K[1]);
                    const int bix = int((b2 - 1) * cv.S[2] + cv.K[2]);
                    const int64_t biv = int64_t(biz) * biy * bix;
                    const int dy_off = int(biv * 128);
                    const size_t lds = size_t(dy_off) + size_t(bov + 1) * 128;
                    if (lds > kLds) continue;
                    double eff = 1.0;
                    const int64_t bo[3] = {b0, b1, b2};
                    for (int k = 0; k < 3; ++k) eff *= double(cv.O[k]) / double(ceil_div(cv.O[k], bo[k]) * bo[k]);
                    const double cost = (double(biv) / bov + 1.0) / eff + 64.0 / bov;
                    if (cost < best) {
                        best = cost;
                        a.BO[0] = b0;
                        a.BO[1] = b1;
                        a.BO[2] = b2;
                        a.biz = biz;
                        a.biy = biy;
                        a.bix = bix;
                        a.dy_off = dy_off;
                        pl.lds = lds;
                    }
                }
        if (best >= 1e299) return pl;
        a.kdg = tgs;
        a.nmb = int32_t(ceil_div(cv.cout, 32));
        a.ncb = int32_t(ceil_div(t.c, 32));
        a.ntg = int32_t(ceil_div(taps, tgs));
        a.blk = 4 * tpw * 1024;
        pl.kind = 2;
    }
    for (int k = 0; k < 3; ++k) a.NB[k] = int32_t(ceil_div(cv.O[k], a.BO[k]));
    a.nbricks = t.n * int64_t(a.NB[0]) * a.NB[1] * a.NB[2];
    const int64_t groups = int64_t(a.nmb) * a.ncb * a.ntg;
    // at most one round of resident workgroups: a few workgroups past the
    // 512 slots would start only when others finish and double the time
    a.nsplit = int32_t(std::max<int64_t>(1, std::min<int64_t>(a.nbricks, kTargetBlocks / groups)));
    a.nblocks = groups * a.nsplit;
    if (a.nblocks >= (int64_t(1) << 31) || a.nbricks == 0) {
        pl.kind = 0;
        return pl;
    }
    pl.a = a;
    return pl;
}

size_t tiled_workspace(const PlanW& pl)
{
    if (pl.kind == 0) return 0;
    return size_t(pl.a.nblocks) * size_t(pl.a.blk) * sizeof(float);
}

template <typename K>
hipError_t launch_with_lds(K fn, const PlanW& pl, hipStream_t s)
{
    const size_t lds = pl.lds;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       int(lds));
    if (e != hipSuccess) return e;
    WgArgs a = pl.a;
    void* args[] = {&a};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(a.nblocks)), dim3(kThreads), args, lds, s);
}

// The pipelined bf16 kernel takes 16-byte loads of every 8-channel group and at
// most kPipeBXU / kPipeBDU staging units per thread.
bool bf16_pipe_ok(const PlanW& pl)
{
    const WgArgs& a = pl.a;
    const int nci = (4 / pl.wco) * 16, nco = pl.wco * 16;
    const int64_t bov = int64_t(a.BO[0]) * a.BO[1] * a.BO[2];
    const int64_t nxu = int64_t(a.biz) * a.biy * ((a.bix + 3) / 4) * (nci / 8);
    const int64_t ndu = (bov / 4) * (nco / 8);
    return a.xvec && a.dvec && a.cin % 8 == 0 && a.cout % 8 == 0 && bov % 4 == 0 && a.BO[2] % 4 == 0 &&
           nxu <= int64_t(kPipeBXU) * kThreads && ndu <= int64_t(kPipeBDU) * kThreads;
}

// The row-pair kernel: 16 input channels, output channels in whole blocks of
// 64, unit stride, one kd plane per tap group (a folded halo on any axes, from
// 16-byte aligned slabs, as the alignment checks require), tile and dy of
// < 4 GiB per batch item, packed coordinates in range, the brick of its own
// shape (W extent a multiple of 16, an even number of K steps) and staging
// within its instruction budget and two workgroups' LDS per CU.
template <int K1, int K2>
hipError_t launch_bf16_pr(const PlanW& pl, hipStream_t s)
{
    const WgArgs& a = pl.a;
    const PrLayout L = pr_layout(a);
    auto fn = a.fold.mask ? &wgrad_bf16_pr<K1, K2, true> : &wgrad_bf16_pr<K1, K2, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       L.bytes);
    if (e != hipSuccess) return e;
    WgArgs aa = a;
    int rp = L.rp, dyo = L.dy_off, bufb = L.bufb;
    uint32_t xbu = uint32_t(a.P[0] * a.P[1] * a.P[2] * a.cin * 2);
    uint32_t dbu = uint32_t(a.O[0] * a.O[1] * a.O[2] * a.cout * 2);
    void* args[] = {&aa, &rp, &dyo, &bufb, &xbu, &dbu};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(aa.nblocks)), dim3(kThreads), args,
                           size_t(L.bytes), s);
}

bool bf16_pr_ok(const PlanW& pl)
{
    const WgArgs& a = pl.a;
    const PrLayout L = pr_layout(a);
    const int64_t bov = int64_t(a.BO[0]) * a.BO[1] * a.BO[2];
    const int64_t xb = a.P[0] * a.P[1] * a.P[2] * a.cin * 2, db = a.O[0] * a.O[1] * a.O[2] * a.cout * 2;
    return pl.kdg == 1 && pl.wco == 4 && a.cin == 16 && a.cout % 64 == 0 && a.S[0] == 1 && a.S[1] == 1 &&
           a.S[2] == 1 && a.xvec && a.dvec && a.K[2] <= 5 && xb < (int64_t(1) << 32) - 64 &&
           db < (int64_t(1) << 32) - 64 && a.BO[2] % 16 == 0 && bov % 32 == 0 && L.rp < 512 && a.biy < 1024 &&
           a.biz < 1024 && a.BO[2] < 512 && a.BO[1] < 1024 && a.BO[0] < 512 && a.biz == a.BO[0] &&
           a.biz * a.biy * L.rp * 2 <= kTrXU * kThreads && bov * 8 <= kTrDU * kThreads && L.bytes <= 80 * 1024;
}

template <int KDG, int K1, int K2, int WCO>
hipError_t launch_bf16_t(const PlanW& pl, hipStream_t s)
{
    if constexpr (KDG == 1 && WCO == 4 && K2 <= 5)
        if (!force_tiled() && bf16_pr_ok(pl)) return launch_bf16_pr<K1, K2>(pl, s);
    if (!bf16_pipe_ok(pl)) return launch_with_lds(&wgrad_bf16_tiled<KDG, K1, K2, WCO>, pl, s);
    const WgArgs& a = pl.a;
    const int64_t nxu = int64_t(a.biz) * a.biy * ((a.bix + 3) / 4) * ((4 / WCO) * 2);
    const int64_t ndu = int64_t(a.BO[0]) * a.BO[1] * a.BO[2] / 4 * (WCO * 2);
    const bool x1 = nxu <= kThreads, d1 = ndu <= kThreads;
    if (x1 && d1) return launch_with_lds(&wgrad_bf16_pipe<KDG, K1, K2, WCO, 1, 1>, pl, s);
    if (x1) return launch_with_lds(&wgrad_bf16_pipe<KDG, K1, K2, WCO, 1, 2>, pl, s);
    if (d1) return launch_with_lds(&wgrad_bf16_pipe<KDG, K1, K2, WCO, 2, 1>, pl, s);
    // two units of each would not fit the registers of two waves per SIMD
    return launch_with_lds(&wgrad_bf16_tiled<KDG, K1, K2, WCO>, pl, s);
}

// The direct-load fp32 kernel: no folded halo (a load instruction has one
// source buffer), 16-byte aligned channel groups, tile and dy of < 4 GiB per
// batch item (32-bit offsets), brick extents below 1024, staging within its
// instruction budget and two workgroups' LDS per compute unit.
hipError_t launch_f32(const Tile3& t, const Conv3& cv, const PlanW& pl, hipStream_t s)
{
    const WgArgs& a = pl.a;
    const int64_t xb = t.P[0] * t.P[1] * t.P[2] * t.c * 4, db = cv.O[0] * cv.O[1] * cv.O[2] * cv.cout * 4;
    const DlLayout L = dl_layout(a);
    const int64_t bov = int64_t(a.BO[0]) * a.BO[1] * a.BO[2];
    // a folded halo: margins along axis 0 only, slabs of < 4 GiB per batch item
    const int64_t plane = t.P[1] * t.P[2] * t.c * 4;
    const int64_t fb_lo = t.lo[0] * plane, fb_hi = t.hi[0] * plane;
    const bool fold_ok = !a.fold.mask || (a.fold.mask == 1u && fb_lo < (int64_t(1) << 32) - 64 &&
                                          fb_hi < (int64_t(1) << 32) - 64);
    const bool dl = fold_ok && a.xvec && a.dvec && t.c % 4 == 0 && cv.cout % 4 == 0 && xb < (int64_t(1) << 32) - 64 &&
                    db < (int64_t(1) << 32) - 64 && a.biz < 1024 && a.biy < 1024 && a.bix < 1024 &&
                    dl_round(a.biz * a.biy * a.bix * 8) <= kDlXU * kThreads &&
                    dl_round(int(bov + (bov & 1)) * 8) <= kDlDU * kThreads && bov + 1 <= kDlTab &&
                    L.bytes <= 80 * 1024;
    if (!dl) return launch_with_lds(&wgrad_f32_tiled<7>, pl, s);
    auto fn = a.fold.mask ? &wgrad_f32_dl<7, true> : &wgrad_f32_dl<7, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       L.bytes);
    if (e != hipSuccess) return e;
    WgArgs aa = a;
    int dyo = L.dy_off, tabo = L.tab_off;
    uint32_t xbu = uint32_t(xb), dbu = uint32_t(db), flu = uint32_t(fb_lo), fhu = uint32_t(fb_hi);
    void* args[] = {&aa, &dyo, &tabo, &xbu, &dbu, &flu, &fhu};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(aa.nblocks)), dim3(kThreads), args,
                           size_t(L.bytes), s);
}

hipError_t launch_bf16(const PlanW& pl, hipStream_t s)
{
    const int k = pl.kdg * 100 + pl.k1 * 10 + pl.k2;
    if (pl.wco == 2) {
        switch (k) {
        case 333: return launch_bf16_t<3, 3, 3, 2>(pl, s);
        case 133: return launch_bf16_t<1, 3, 3, 2>(pl, s);
        case 155: return launch_bf16_t<1, 5, 5, 2>(pl, s);
        case 111: return launch_bf16_t<1, 1, 1, 2>(pl, s);
        case 113: return launch_bf16_t<1, 1, 3, 2>(pl, s);
        case 115: return launch_bf16_t<1, 1, 5, 2>(pl, s);
        default: break;
        }
    } else {
        switch (k) {
        case 333: return launch_bf16_t<3, 3, 3, 4>(pl, s);
        case 133: return launch_bf16_t<1, 3, 3, 4>(pl, s);
        case 155: return launch_bf16_t<1, 5, 5, 4>(pl, s);
        case 111: return launch_bf16_t<1, 1, 1, 4>(pl, s);
        case 113: return launch_bf16_t<1, 1, 3, 4>(pl, s);
        case 115: return launch_bf16_t<1, 1, 5, 4>(pl, s);
        default: break;
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace

size_t conv_wgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    return kWgradStatusBytes + std::max({generic_wgrad_workspace(t, cv), tiled_workspace(plan_wgrad(t, cv, dt)),
                                         wgrad_tr_workspace(t, cv, dt), wgrad_xm_workspace(t, cv, dt)});
}

namespace {

__global__ void wgrad_status_clear(uint32_t* status)
{
    // the status word and the zero source (status block bytes 0 .. 127)
    if (threadIdx.x < 32) status[threadIdx.x] = 0u;
}

}  // namespace

hipError_t launch_wgrad_status_clear(uint32_t* status, hipStream_t s)
{
    hipLaunchKernelGGL(wgrad_status_clear, dim3(1), dim3(64), 0, s, status);
    return hipGetLastError();
}

namespace {

// ws: the call's workspace (status block first, see kWgradStatusBytes)
hipError_t run_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy, float* dw,
                     void* ws_all, const Fold* fold, hipStream_t s)
{
    uint32_t* status = static_cast<uint32_t*>(ws_all);
    void* ws = static_cast<char*>(ws_all) + kWgradStatusBytes;
    {
        hipError_t e = launch_wgrad_status_clear(status, s);
        if (e != hipSuccess) return e;
        e = launch_wgrad_xm(t, cv, dt, tile, dy, dw, ws, fold, status, s);
        if (e != hipErrorNotSupported) return e;
    }
    if (!fold) {
        int32_t red[6];
        hipError_t e = launch_wgrad_tr(t, cv, dt, tile, dy, static_cast<float*>(ws), red, s);
        if (e != hipErrorNotSupported) {
            if (e != hipSuccess) return e;
            WgArgs a{};
            a.part = static_cast<float*>(ws);
            a.dw = dw;
            a.cin = t.c;
            a.cout = cv.cout;
            for (int k = 0; k < 3; ++k) a.K[k] = int32_t(cv.K[k]);
            a.nmb = red[0];
            a.ncb = red[1];
            a.ntg = red[2];
            a.blk = red[3];
            a.kdg = red[4];
            a.nsplit = red[5];
            const int64_t total = int64_t(a.nmb) * a.ncb * a.ntg * a.blk;
            const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 1 << 16)));
            int kind = 2, kdg = a.kdg, k1 = 0, k2 = 0, wco = 0;
            void* args[] = {&a, &kind, &kdg, &k1, &k2, &wco};
            return hipLaunchKernel(reinterpret_cast<const void*>(&wgrad_reduce), dim3(grid), dim3(256), args, 0, s);
        }
    }
    PlanW pl = plan_wgrad(t, cv, dt);
    if (pl.kind == 0) return generic_conv_wgrad(t, cv, dt, tile, dy, dw, ws, fold, s);
    pl.a.tile = static_cast<const char*>(tile);
    pl.a.dy = static_cast<const char*>(dy);
    const int64_t esz = dt == SHARD_BF16 ? 2 : 4;
    bool xal = reinterpret_cast<uintptr_t>(tile) % 16 == 0;
    if (fold) {
        pl.a.fold = *fold;
        for (int k = 0; k < 3; ++k)
            for (int sd = 0; sd < 2; ++sd) xal = xal && reinterpret_cast<uintptr_t>(fold->slab[k][sd]) % 16 == 0;
    }
    pl.a.xvec = xal && (t.c * esz) % 16 == 0;
    pl.a.dvec = (reinterpret_cast<uintptr_t>(dy) % 16 == 0) && (cv.cout * esz) % 16 == 0;
    pl.a.part = static_cast<float*>(ws);
    pl.a.dw = dw;
    pl.a.zeros = static_cast<const char*>(ws_all) + kWgradZeroOff;
    hipError_t e = pl.kind == 1 ? launch_bf16(pl, s) : launch_f32(t, cv, pl, s);
    if (e != hipSuccess) return e;
    const int64_t total = int64_t(pl.a.nmb) * pl.a.ncb * pl.a.ntg * pl.a.blk;
    const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 1 << 16)));
    WgArgs a = pl.a;
    int kind = pl.kind, kdg = pl.a.kdg, k1 = pl.k1, k2 = pl.k2, wco = pl.wco;
    void* args[] = {&a, &kind, &kdg, &k1, &k2, &wco};
    return hipLaunchKernel(reinterpret_cast<const void*>(&wgrad_reduce), dim3(grid), dim3(256), args, 0, s);
}

}  // namespace

hipError_t launch_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                             float* dw, void* ws, hipStream_t s)
{
    return run_wgrad(t, cv, dt, tile, dy, dw, ws, nullptr, s);
}

hipError_t launch_conv_wgrad_folded(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                    const void* dy, float* dw, void* ws, const Fold& fold, hipStream_t s)
{
    return run_wgrad(t, cv, dt, tile, dy, dw, ws, &fold, s);
}

}  // namespace shardconv
