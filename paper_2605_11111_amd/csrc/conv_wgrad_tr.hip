// Weight gradient, bf16: dW[co][ci][t] = sum_v dy[v][co] * tile[v*S + t - pad][ci],
// as a persistent split-K implicit GEMM with M = co, N = ci, K = output voxels.
//
// Both operands need 8 consecutive K values (voxels) per lane, while the data is
// channels-last. Instead of transposing while staging, the input footprint and
// dy of a brick are copied to LDS unchanged (channels-last, direct global->LDS
// buffer loads, double buffered) and every operand is read with
// ds_read_b64_tr_b16: within each group of 16 lanes, lane i addresses voxel
// row k0 + i/4 at channels c0 + 4*(i%4), and lane j receives channel c0 + j of
// voxels k0..k0+3. Two such reads give a v_mfma_f32_32x32x16_bf16 operand.
// Since every lane forms its own address, a tap offset or a stride is just a
// different voxel row: no alignment constraint, no shuffles.
//
// The four waves split the taps of a tap group (wave w: taps w, w+4, ...); all
// share the dy operand. Each workgroup keeps its 32x32 dW tiles in registers
// over its bricks and writes them once; the split-K sum runs in a fixed order
// in wgrad_reduce, so results are bit-identical run to run.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t2;
typedef __attribute__((ext_vector_type(4))) short s16x4_t2;
typedef __attribute__((ext_vector_type(16))) float f32x16_t2;

#define SC_LDS2(p) ((__attribute__((address_space(3))) void*)(p))

namespace {

struct TrArgs {
    const char* tile;
    const char* dy;
    float* part;
    int64_t n, cin, cout;
    int64_t P[3], O[3];
    int32_t K[3], S[3], pad[3];
    int32_t NB[3];
    int64_t nbricks;
    uint32_t tile_bytes, dy_bytes;  // per batch item (< 2^32)
    int32_t nmb, ncb, ntg, tgs;     // channel blocks, tap groups, taps per group
    int32_t nsplit;                 // workgroups per group; split s takes bricks s, s + nsplit, ...
};

template <int BZ, int BY, int BX, int KD, int KH, int KW, int SD, int SH, int SW, int TPW>
struct TrCfg {
    static constexpr int BOV = BZ * BY * BX;
    static constexpr int BIZ = (BZ - 1) * SD + KD, BIY = (BY - 1) * SH + KH, BIX = (BX - 1) * SW + KW;
    static constexpr int BIV = BIZ * BIY * BIX;
    static constexpr int X_SLOTS = BIV * 4;                     // 4 x 16 B per voxel (32 channels)
    static constexpr int X_SLOTS_PAD = (X_SLOTS + 63) / 64 * 64;
    static constexpr int DY_SLOTS = BOV * 4;
    static constexpr int SLOTS = X_SLOTS_PAD + DY_SLOTS;
    static constexpr int NIT = (SLOTS + 255) / 256;
    static constexpr int X_BYTES = X_SLOTS_PAD * 16;
    static constexpr int STAGE_BYTES = SLOTS * 16;
    static constexpr int LDS_BYTES = 2 * STAGE_BYTES;
};


template <int BZ, int BY, int BX, int KD, int KH, int KW, int SD, int SH, int SW, int TPW>
__global__ __launch_bounds__(256, 1) void wgrad_tr(TrArgs a)
{
    using C = TrCfg<BZ, BY, BX, KD, KH, KW, SD, SH, SW, TPW>;
    static_assert(BX % 16 == 0, "a 16-voxel K step must stay inside one W row");
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t G = gridDim.x;

    // logical index: group innermost, so each XCD holds a contiguous range of splits per group
    const int64_t Lg = xcd_remap(blockIdx.x, G);
    const int64_t groups = int64_t(a.nmb) * a.ncb * a.ntg;
    int64_t b = Lg % groups;
    const int64_t split = Lg / groups;
    const int tg = int(b % a.ntg);
    b /= a.ntg;
    const int cb = int(b % a.ncb);
    b /= a.ncb;
    const int mb = int(b);
    const int64_t ci0 = int64_t(cb) * 32, co0 = int64_t(mb) * 32;
    constexpr int TAPS = KD * KH * KW;

    const uint32_t lds0 = lds_addr(lds);
    // this wave's taps (w, w + 4, ...) as byte offsets of their voxel shift in the input brick
    int toff[TPW];
    bool tok[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tl = wave + 4 * i;
        const int t = tg * a.tgs + tl;
        tok[i] = tl < a.tgs && t < TAPS;
        const int tt = tok[i] ? t : 0;
        const int kw = tt % KW, kh = (tt / KW) % KH, kd = tt / (KW * KH);
        toff[i] = ((kd * C::BIY + kh) * C::BIX + kw) * 64;
    }

    // per-thread staging slots, brick invariant: relative byte offset and packed coordinates
    uint32_t srel[C::NIT], szyx[C::NIT];
#pragma unroll
    for (int it = 0; it < C::NIT; ++it) {
        const int s = it * 256 + tid;
        if (s < C::X_SLOTS) {
            const int u = s & 3, v = s >> 2;
            const int x = v % C::BIX, yz = v / C::BIX, y = yz % C::BIY, z = yz / C::BIY;
            srel[it] = uint32_t((((int64_t(z) * a.P[1] + y) * a.P[2] + x) * a.cin + ci0 + 8 * u) * 2);
            szyx[it] = (uint32_t(z) << 20) | (uint32_t(y) << 10) | uint32_t(x) | (uint32_t(u) << 29);
        } else if (s >= C::X_SLOTS_PAD && s < C::SLOTS) {
            const int sd = s - C::X_SLOTS_PAD;
            const int u = sd & 3, f = sd >> 2;
            const int x = f % BX, y = (f / BX) % BY, z = f / (BX * BY);
            srel[it] = uint32_t((((int64_t(z) * a.O[1] + y) * a.O[2] + x) * a.cout + co0 + 8 * u) * 2);
            szyx[it] = (uint32_t(z) << 20) | (uint32_t(y) << 10) | uint32_t(x) | (uint32_t(u) << 29) | (1u << 31);
        } else {
            srel[it] = 0;
            szyx[it] = 0xffffffffu;  // padding slot: no load
        }
    }

    // tr-read lane terms: voxel k0 + i/4 and channel c0 + 4*(i%4) of the lane's 16-lane group
    const int kl = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int colb = (16 * ((lane >> 4) & 1) + 4 * (lane & 3)) * 2;

    f32x16_t2 acc[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;

    auto stage = [&](int64_t br, int buf) {
        int64_t bb = br;
        const int bx = int(bb % a.NB[2]);
        bb /= a.NB[2];
        const int by = int(bb % a.NB[1]);
        bb /= a.NB[1];
        const int bz = int(bb % a.NB[0]);
        const int64_t nn = bb / a.NB[0];
        const int64_t o0 = int64_t(bz) * BZ, o1 = int64_t(by) * BY, o2 = int64_t(bx) * BX;
        const int64_t i0 = o0 * SD - a.pad[0], i1 = o1 * SH - a.pad[1], i2 = o2 * SW - a.pad[2];
        const bool xin = i0 >= 0 && i0 + C::BIZ <= a.P[0] && i1 >= 0 && i1 + C::BIY <= a.P[1] && i2 >= 0 &&
                         i2 + C::BIX <= a.P[2] && ci0 + 32 <= a.cin;
        const bool din = o0 + BZ <= a.O[0] && o1 + BY <= a.O[1] && o2 + BX <= a.O[2] && co0 + 32 <= a.cout;
        const int64_t xorg = ((i0 * a.P[1] + i1) * a.P[2] + i2) * a.cin * 2;
        const int64_t dorg = ((o0 * a.O[1] + o1) * a.O[2] + o2) * a.cout * 2;
        __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.tile) + nn * int64_t(a.tile_bytes), short(0), int(a.tile_bytes), 0x00020000);
        __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.dy) + nn * int64_t(a.dy_bytes), short(0), int(a.dy_bytes), 0x00020000);
        char* dst = lds + buf * C::STAGE_BYTES;
#pragma unroll
        for (int it = 0; it < C::NIT; ++it) {
            const uint32_t zyx = szyx[it];
            if (zyx == 0xffffffffu) continue;
            const int64_t z = (zyx >> 20) & 511, y = (zyx >> 10) & 1023, x = zyx & 1023;
            const int64_t u = (zyx >> 29) & 3;
            char* d = dst + (it * 256 + wave * 64) * 16;
            if (!(zyx >> 31)) {
                uint32_t off;
                if (xin) {
                    off = uint32_t(xorg + srel[it]);
                } else {
                    const int64_t t0 = i0 + z, t1 = i1 + y, t2 = i2 + x;
                    const bool ok = t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2] &&
                                    ci0 + 8 * u < a.cin;
                    off = ok ? uint32_t(xorg + int64_t(srel[it])) : a.tile_bytes;
                }
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, SC_LDS2(d), 16, off, 0, 0, 0);
            } else {
                uint32_t off;
                if (din) {
                    off = uint32_t(dorg + srel[it]);
                } else {
                    const bool ok = o0 + z < a.O[0] && o1 + y < a.O[1] && o2 + x < a.O[2] && co0 + 8 * u < a.cout;
                    off = ok ? uint32_t(dorg + int64_t(srel[it])) : a.dy_bytes;
                }
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, SC_LDS2(d), 16, off, 0, 0, 0);
            }
        }
    };

    // operand reads of K step ks (16 output voxels) from stage buffer xs / ds. Every
    // wave issues 2 + 2 * TPW reads per step (a wave with fewer taps reads tap 0
    // again) so that the lgkmcnt waits below are the same for all waves.
    auto load_step = [&](uint32_t xs, uint32_t ds, int ks, lds_u32x4& av, lds_u32x4 (&bv)[TPW]) {
        const int f = 16 * ks + kl;
        const int xo = f % BX, yo = (f / BX) % BY, zo = f / (BX * BY);
        const int vin = ((zo * SD) * C::BIY + yo * SH) * C::BIX + xo * SW;
        const uint2 a0 = lds_read_tr16_b64(ds + uint32_t(f * 64 + colb));
        const uint2 a1 = lds_read_tr16_b64(ds + uint32_t((f + 4) * 64 + colb));
        av = lds_u32x4{a0.x, a0.y, a1.x, a1.y};
        const uint32_t xb0 = xs + uint32_t(vin * 64 + colb);
        const uint32_t xb1 = xb0 + uint32_t(4 * SW * 64);  // f + 4 stays in the same W row (BX % 16 == 0)
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const uint2 b0 = lds_read_tr16_b64(xb0 + uint32_t(toff[i]));
            const uint2 b1 = lds_read_tr16_b64(xb1 + uint32_t(toff[i]));
            bv[i] = lds_u32x4{b0.x, b0.y, b1.x, b1.y};
        }
    };
    // LDS operations per step (the wait allows at most 15 outstanding)
    constexpr int RPS = 2 + 2 * TPW;
    constexpr int WAIT_NEXT = RPS < 15 ? RPS : 15;
    auto ready = [&](lds_u32x4& av, lds_u32x4 (&bv)[TPW]) {
        lds_ready(av);
#pragma unroll
        for (int i = 0; i < TPW; ++i) lds_ready(bv[i]);
    };
    auto mfma_step = [&](const lds_u32x4& av, const lds_u32x4 (&bv)[TPW]) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            if (!tok[i]) continue;
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t2, av),
                                                             __builtin_bit_cast(bf16x8_t2, bv[i]), acc[i], 0, 0, 0);
        }
    };

    int64_t b_cur = split;
    if (b_cur < a.nbricks) stage(b_cur, 0);
    wait_vm_barrier<0>();
    int buf = 0;
    while (b_cur < a.nbricks) {
        const int64_t b_next = b_cur + a.nsplit;
        if (b_next < a.nbricks) stage(b_next, buf ^ 1);
        const uint32_t xs = lds0 + uint32_t(buf * C::STAGE_BYTES);
        const uint32_t ds = xs + uint32_t(C::X_BYTES);
        // software pipeline: the operands of step ks + 1 are read while step ks multiplies
        constexpr int NKS = C::BOV / 16;
        lds_u32x4 av[2], bv[2][TPW];
        load_step(xs, ds, 0, av[0], bv[0]);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int cb = ks & 1;
            if (ks + 1 < NKS) {
                load_step(xs, ds, ks + 1, av[cb ^ 1], bv[cb ^ 1]);
                lds_wait<WAIT_NEXT>();
            } else {
                lds_wait<0>();
            }
            ready(av[cb], bv[cb]);
            mfma_step(av[cb], bv[cb]);
        }
        wait_vm_barrier<0>();
        buf ^= 1;
        b_cur = b_next;
    }
    // partial tile: [wave][tap i][lane][16]
    const int64_t grp = (int64_t(mb) * a.ncb + cb) * a.ntg + tg;

    float4* out = reinterpret_cast<float4*>(a.part + (split * groups + grp) * int64_t(4 * TPW * 1024) +
                                            int64_t(wave) * TPW * 1024);
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            out[(i * 64 + lane) * 4 + r4] =
                make_float4(acc[i][4 * r4], acc[i][4 * r4 + 1], acc[i][4 * r4 + 2], acc[i][4 * r4 + 3]);
}

}  // namespace

// The transpose-read weight gradient applies to bf16 with channel counts that
// are multiples of 8, per-batch tile and dy sizes below 4 GiB, 16-byte aligned
// buffers and the kernel/stride/brick shapes instantiated here.
struct TrPlan {
    bool ok;
    int cfg;  // 0: 3D 3x3x3 unit stride, brick 2x4x32; 1: 2D 3x3 unit stride, brick 1x8x32
    TrArgs a;
    size_t lds;
    int64_t grid;
};

constexpr int kTrTPW = 7;

static TrPlan plan_tr(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    TrPlan p{};
    p.ok = false;
    if (force_generic() || force_tiled() || dt != SHARD_BF16 || t.c % 8 != 0 || cv.cout % 8 != 0) return p;
    const int64_t tb = t.P[0] * t.P[1] * t.P[2] * t.c * 2;
    const int64_t db = cv.O[0] * cv.O[1] * cv.O[2] * cv.cout * 2;
    if (tb >= (int64_t(1) << 32) - 64 || db >= (int64_t(1) << 32) - 64) return p;
    for (int k = 0; k < 3; ++k)
        if (cv.S[k] != 1 || std::abs(cv.pad[k]) > (1 << 20) || cv.O[k] > (int64_t(1) << 30)) return p;
    int bz, by, bx;
    size_t lds;
    if (cv.K[0] == 3 && cv.K[1] == 3 && cv.K[2] == 3) {
        p.cfg = 0;
        bz = 2, by = 4, bx = 32;
        lds = TrCfg<2, 4, 32, 3, 3, 3, 1, 1, 1, kTrTPW>::LDS_BYTES;
    } else if (cv.K[0] == 1 && cv.K[1] == 3 && cv.K[2] == 3) {
        p.cfg = 1;
        bz = 1, by = 8, bx = 32;
        lds = TrCfg<1, 8, 32, 1, 3, 3, 1, 1, 1, kTrTPW>::LDS_BYTES;
    } else {
        return p;
    }
    TrArgs& a = p.a;
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
    a.NB[0] = int32_t(ceil_div(cv.O[0], bz));
    a.NB[1] = int32_t(ceil_div(cv.O[1], by));
    a.NB[2] = int32_t(ceil_div(cv.O[2], bx));
    a.nbricks = t.n * int64_t(a.NB[0]) * a.NB[1] * a.NB[2];
    if (a.nbricks == 0) return p;
    a.tile_bytes = uint32_t(tb);
    a.dy_bytes = uint32_t(db);
    a.nmb = int32_t(ceil_div(cv.cout, 32));
    a.ncb = int32_t(ceil_div(t.c, 32));
    a.tgs = 4 * kTrTPW;
    a.ntg = int32_t(ceil_div(cv.taps(), a.tgs));
    const int64_t groups = int64_t(a.nmb) * a.ncb * a.ntg;
    a.nsplit = int32_t(std::max<int64_t>(1, std::min<int64_t>(a.nbricks, ceil_div(256, groups))));
    if (a.nsplit >= 8) a.nsplit -= a.nsplit % 8;
    p.grid = groups * a.nsplit;
    p.lds = lds;
    p.ok = p.grid < (int64_t(1) << 31);
    return p;
}

size_t wgrad_tr_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    const TrPlan p = plan_tr(t, cv, dt);
    if (!p.ok) return 0;
    return size_t(p.grid) * 4 * kTrTPW * 1024 * sizeof(float);
}

// Launches the tr kernel and fills the reduce description {nmb, ncb, ntg,
// floats per block, taps per group, nsplit}. Returns hipErrorNotSupported when
// it does not apply.
hipError_t launch_wgrad_tr(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* part, int32_t red[6], hipStream_t s)
{
    TrPlan p = plan_tr(t, cv, dt);
    if (!p.ok || reinterpret_cast<uintptr_t>(tile) % 16 != 0 || reinterpret_cast<uintptr_t>(dy) % 16 != 0)
        return hipErrorNotSupported;
    p.a.tile = static_cast<const char*>(tile);
    p.a.dy = static_cast<const char*>(dy);
    p.a.part = part;
    const void* fn = p.cfg == 0 ? reinterpret_cast<const void*>(&wgrad_tr<2, 4, 32, 3, 3, 3, 1, 1, 1, kTrTPW>)
                                : reinterpret_cast<const void*>(&wgrad_tr<1, 8, 32, 1, 3, 3, 1, 1, 1, kTrTPW>);
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(p.lds));
    if (e != hipSuccess) return e;
    void* args[] = {&p.a};
    e = hipLaunchKernel(fn, dim3(unsigned(p.grid)), dim3(256), args, p.lds, s);
    red[0] = p.a.nmb;
    red[1] = p.a.ncb;
    red[2] = p.a.ntg;
    red[3] = 4 * kTrTPW * 1024;
    red[4] = p.a.tgs;
    red[5] = p.a.nsplit;
    return e;
}

}  // namespace shardconv
