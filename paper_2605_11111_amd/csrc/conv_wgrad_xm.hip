// Weight gradient, bf16, unit stride, 3 x 3 taps in H and W (KD = 1 or 3):
// dW[co][ci][kd][kh][kw] = sum over output voxels v of dy[v][co] * tile[v + t - pad][ci],
// a split-K implicit GEMM with M = 32 output channels, N = 32 input channels and
// K = output voxels along W, on v_mfma_f32_32x32x16_bf16.
//
//  * Wave roles: each role is one (Co tile, Ci tile, kd) and owns the nine
//    (kh, kw) taps of that plane offset as nine 32 x 32 fp32 accumulators kept in
//    registers over all the workgroup's bricks. With four roles (one wave each)
//    every wave also issues a quarter of the staging loads, one per MFMA group.
//    With three roles the workgroup has eight waves, two per SIMD: the two waves
//    of a role's SIMD split the tile's K (voxels) in halves - each keeps its own
//    accumulators, summed later with the other partials - and the fourth SIMD's
//    two waves only issue the staging loads. A direct global->LDS load stalls its
//    wave at issue for tens of cycles; with two MFMA waves per SIMD the other one
//    keeps the matrix core busy meanwhile, and no compute wave issues loads.
//  * A workgroup owns bricks of BZ x BY output rows and marches along W in
//    32-voxel tiles. Each tile's inputs (dy rows and the BZ+KD-1 x BY+2 input rows:
//    32 voxels in a main area, the next 4 in a halo area) are staged unchanged
//    (channels-last) by direct global->LDS buffer loads, double buffered;
//    out-of-range offsets load zeros.
//  * Operands need 8 consecutive voxels per lane; they are read with
//    ds_read_b64_tr_b16 (transpose on read). K step s of lane half g covers
//    voxels 16g + 8s .. + 7, so a lane holds the contiguous run 16g .. 16g + 19
//    of its channel after five reads, and the W taps are register selections:
//    kw = 0 and 2 are dword-aligned windows, kw = 1 is one v_alignbit per dword.
//    One row's five reads serve all three kw of both K steps (a wave that owns
//    one K step reads the three that cover its 10-voxel run).
//  * Walking the brick's output rows along H, input row y + kh serves output
//    rows y, y - 1, y - 2: each input row is read once per plane (a ring of four
//    register slots per plane parity), so a wave issues about nine 512-byte
//    transposed reads per eighteen MFMAs (five per nine with one K step).
//  * The partial of every workgroup is written once; wgrad_xm_reduce1/2 sum the
//    partials in a fixed order (results are bitwise repeatable).
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_w;
typedef __attribute__((ext_vector_type(16))) float f32x16_w;

#define SC_LDSW(p) ((__attribute__((address_space(3))) void*)(p))

namespace {

struct WxArgs {
    const char* tile;
    const char* dy;
    float* part;
    int32_t P[3], O[3];
    int32_t pad[3];
    int32_t NBZ, NBY, NXT;  // bricks along D and H, 32-voxel tiles along W
    int32_t TZ, TY;         // raster block of TZ x TY bricks (divides NBZ x NBY)
    int32_t nseg, T;        // W segments per brick row and their length in tiles
    uint32_t nbricks;       // n * NBZ * NBY * nseg
    uint32_t tile_bytes, dy_bytes;  // per batch item (< 2^32)
    uint32_t xrow, xplane, yrow, yplane;  // byte strides of tile and dy rows and planes
    // halo folded into the loads along axis fa (0 or 1): padded rows c < flo come
    // from fslab[0], rows c >= fhi from fslab[1] (null: zero), the rest from the tile
    const char* fslab[2];
    uint32_t fbatch[2];  // slab bytes per batch item
    uint32_t fSZ[2];     // slab stride along axis 0, bytes
    int32_t fa, flo, fhi;
    uint32_t* status;     // the call's status word (nonzero: a hand-off wait gave up)
    uint32_t wait_polls;  // poll bound of a hand-off wait
};

// 16-byte unit swizzle of staged voxel v for UPV units per voxel: with 128-byte
// voxels the four rows of a transposed read would fall on two bank windows, so
// rows with bit 1 set move by 32 bytes.
template <int UPV>
__device__ __forceinline__ constexpr int wx_swz(int v)
{
    return UPV == 8 ? (((v >> 1) & 1) << 1) : 0;
}

template <int KD, int NCI, int NCO, int BZ, int BY>
struct WxCfg {
    static constexpr int CIN = 32 * NCI, COUT = 32 * NCO;
    static constexpr int UPX = CIN / 8, UPY = COUT / 8;   // 16-byte units per voxel
    static constexpr int NR = NCO * NCI * KD;             // wave roles
    static_assert(NR >= 1 && NR <= 4, "at most four roles per workgroup");
    static constexpr int XRZ = BZ + KD - 1, XRY = BY + 2, XR = XRZ * XRY;
    // input row r: voxels 0..31 in the main area, voxels 32..35 in the halo area
    static constexpr int XROW = 32 * UPX * 16;
    static constexpr int IPR_X = 32 * UPX / 64;            // direct-load instructions per main row
    static constexpr int XH_ROW = 4 * UPX * 16;
    static constexpr int XH_SLOTS = XR * 4 * UPX;
    static_assert(XH_SLOTS % 64 == 0, "whole halo instructions");
    static constexpr int XH_INSTR = XH_SLOTS / 64;
    static constexpr int X_BYTES = XR * XROW;
    static constexpr int XH_BYTES = XH_SLOTS * 16;
    static constexpr int YROW = 32 * UPY * 16;
    static constexpr int IPR_Y = 32 * UPY / 64;
    static constexpr int Y_BYTES = BZ * BY * YROW;
    static constexpr int X_INSTR = XR * IPR_X, Y_INSTR = BZ * BY * IPR_Y;
    static constexpr int N_INSTR = X_INSTR + XH_INSTR + Y_INSTR;
    static constexpr int STAGE_BYTES = X_BYTES + XH_BYTES + Y_BYTES;
    static constexpr int LDS_BYTES = 2 * STAGE_BYTES;
    static constexpr int NQ = BZ * BY;                     // output rows per tile
    static constexpr int PART_FLOATS = 4 * 9 * 1024;       // per K split of a workgroup: [role][tap][lane][16]
};

// KS = 1: four waves, two stage buffers, a workgroup barrier per tile.
// KS = 2: eight waves, K split in halves between the two waves of a SIMD (three
// roles only), NB stage buffers handed between loaders and compute waves through
// LDS counters instead of barriers (see the flag protocol below).
template <int KD, int NCI, int NCO, int BZ, int BY, int KS, int NB, bool FOLD>
__global__ __launch_bounds__(256 * KS, 1) void wgrad_xm(WxArgs a)
{
    using C = WxCfg<KD, NCI, NCO, BZ, BY>;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63;
    // wave w runs on SIMD w % 4; ks = w / 4 is its K half (KS = 2)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int simd = wave & 3, ks = wave >> 2;
    const uint32_t G = gridDim.x;
    const uint32_t L = uint32_t(xcd_remap(blockIdx.x, G));
    // With four roles every wave computes and issues a quarter of the staging
    // loads; with three, the waves of SIMD 3 are dedicated loaders that issue
    // them all (their stalls at issue then never hold back a matrix core).
    static_assert(C::NR == 3 || C::NR == 4, "three or four wave roles");
    static_assert(KS == 1 || (KS == 2 && C::NR == 3), "K split only with three roles");
    constexpr bool kLoader = C::NR == 3;
    const int role = simd < C::NR ? simd : 0;
    const int kd = role % KD, cb = (role / KD) % NCI, mb = role / (KD * NCI);
    const uint32_t lds0 = lds_addr(lds);
    static_assert(KS == 1 ? NB == 2 : (NB >= 2 && NB <= 4), "stage buffers");

    // Flag protocol (KS = 2). After the NB stage buffers LDS holds two counters
    // per buffer b: full[b], raised by each of the two loader waves once the
    // loads of a unit it issued into b have landed, and free[b], raised by each of
    // the six compute waves once it has read a unit out of b. Unit u lives in
    // buffer u % NB and is that buffer's (u / NB + 1)-th fill: a compute wave
    // starts it when full[b] >= 2 (u / NB + 1), and a loader refills b for unit u
    // when free[b] >= 6 (u / NB). Neither wait depends on a later signal of the
    // waiting wave's own kind, so the pipeline cannot deadlock. Every wait is also
    // bounded: a wait that gives up (a.wait_polls polls, by default 2^20, far
    // beyond any real wait) raises an abort word that ends every later wait at
    // once, so a broken hand-off never hangs the kernel; it also sets the call's
    // status word in global memory, and the reduction then writes NaN into every
    // dw element, so the broken result cannot pass for a correct one.
    constexpr int NCW = 3 * KS;  // compute waves (KS = 2)
    const uint32_t flag_full0 = lds0 + uint32_t(NB * C::STAGE_BYTES);
    const uint32_t flag_free0 = flag_full0 + uint32_t(4 * NB);
    const uint32_t flag_abort = flag_free0 + uint32_t(4 * NB);
    if (KS == 2) {
        if (tid < 2 * NB + 1) reinterpret_cast<uint32_t*>(lds + NB * C::STAGE_BYTES)[tid] = 0u;
        __syncthreads();
    }
    auto raise = [&](uint32_t addr) {
        if (lane == 0) lds_add_u32(addr, 1u);
    };
    auto spin_until = [&](uint32_t addr, uint32_t target) {
        for (uint32_t it = 0; it < a.wait_polls; ++it) {
            if (lds_read_u32_now(addr) >= target || lds_read_u32_now(flag_abort) != 0u) return;
            __builtin_amdgcn_s_sleep(1);
        }
        raise(flag_abort);
        // a vector atomic from one lane (the status word is read after the kernel)
        if (lane == 0) __hip_atomic_fetch_or(a.status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };

    // ---- staging (loader waves) ----
    // a brick's rows (bz, by) and batch item nn are decoded once per brick
    struct Pos {
        uint32_t brick;
        int32_t j, jend;
        int32_t bz, by;
        uint32_t nn;
    };
    auto seg_start = [&](Pos& p) {
        if (p.brick >= a.nbricks) return;
        const uint32_t t = p.brick / uint32_t(a.nseg);
        const int32_t seg = int32_t(p.brick - t * uint32_t(a.nseg));
        p.j = seg * a.T;
        p.jend = min(p.j + a.T, a.NXT);
        brick_rows(t, a.NBZ, a.NBY, a.TZ, a.TY, p.bz, p.by, p.nn);
    };
    auto advance = [&](Pos& p) {
        if (++p.j >= p.jend) {
            p.brick += G;
            seg_start(p);
        }
    };
    // One 16-byte x load of padded voxel row (z, y) at tile offset `off` (the
    // offset of that row in the padded tile): with the halo folded, a row in a
    // margin along the fold axis comes from its slab (the offset moved to the
    // slab's layout), zero past the data. (z, y) may differ between lanes (the
    // halo area packs several rows per instruction): the branch then diverges
    // and each lane's load runs under its own source, writing only its own slot.
    auto slab_rsrc = [&](int sd, uint32_t nn) {
        return __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.fslab[sd] ? a.fslab[sd] + int64_t(nn) * a.fbatch[sd] : a.tile), short(0),
            a.fslab[sd] ? int(a.fbatch[sd]) : 0, 0x00020000);
    };
    // A unit whose staged rows all lie inside [flo, fhi) along the fold axis takes
    // the plain loads (`touch` false, uniform over the unit).
    auto touches = [&](int32_t z0, int32_t y0) {
        const int32_t c0 = a.fa == 0 ? z0 : y0, n = a.fa == 0 ? C::XRZ : C::XRY;
        return FOLD && (c0 < a.flo || c0 + n > a.fhi);
    };
    auto xload = [&](__amdgpu_buffer_rsrc_t rt, __amdgpu_buffer_rsrc_t rl, __amdgpu_buffer_rsrc_t rh, char* dst,
                     uint32_t off, bool ok, int32_t z, int32_t y, bool touch) {
        if (!FOLD || !touch) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rt, SC_LDSW(dst), 16, ok ? off : 0xFFFFFFC0u, 0, 0, 0);
            return;
        }
        const int32_t c = a.fa == 0 ? z : y;
        if (c < a.flo) {
            const uint32_t o = off - uint32_t(z) * (a.xplane - a.fSZ[0]);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, SC_LDSW(dst), 16, ok ? o : 0xFFFFFFC0u, 0, 0, 0);
        } else if (c >= a.fhi) {
            const uint32_t o = off - uint32_t(z) * (a.xplane - a.fSZ[1]) -
                               uint32_t(a.fhi) * (a.fa == 0 ? a.xplane : a.xrow);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rh, SC_LDSW(dst), 16, ok ? o : 0xFFFFFFC0u, 0, 0, 0);
        } else {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rt, SC_LDSW(dst), 16, ok ? off : 0xFFFFFFC0u, 0, 0, 0);
        }
    };

    // Staging: wave w loads the input rows r = w, w + 4, ... (IPR_X instructions
    // each), the halo instructions h = w, w + 4, ... and the dy rows w, w + 4, ...
    // Main and dy rows: lane l carries unit l % UPV of voxel piece * (64 / UPV) +
    // l / UPV; halo area: 4 * UPX lanes per row, unit l % UPX of voxel 32 + (l / UPX) % 4.
    // Byte offsets are 32-bit (a batch item is < 4 GiB; only in-range offsets are
    // used, so wrap-around in the intermediate sums is harmless).
    const int vx = lane / C::UPX, ux = lane % C::UPX;
    const int vy = lane / C::UPY, uy = lane % C::UPY;
    const int hrow = lane / (4 * C::UPX), hv = 32 + (lane / C::UPX) % 4;
    static_assert((64 / C::UPX) % 4 == 0 && (64 / C::UPY) % 4 == 0, "swizzle bit is lane-constant");
    const uint32_t lxm = uint32_t(vx * C::CIN * 2 + (ux ^ wx_swz<C::UPX>(vx)) * 16);
    const uint32_t lym = uint32_t(vy * C::COUT * 2 + (uy ^ wx_swz<C::UPY>(vy)) * 16);
    const uint32_t lxh = uint32_t(hv * C::CIN * 2 + (ux ^ wx_swz<C::UPX>(hv)) * 16);
    constexpr int XPI = 64 / C::UPX, YPI = 64 / C::UPY;  // voxels per instruction
    constexpr int HRPI = 64 / (4 * C::UPX);              // halo rows per instruction
    // A unit's staging is a set-up (its uniform values, once per tile) and the
    // wave's single loads k = 0 .. KLOADS - 1, which the main loop spreads over the
    // first rows of the tile: issued as one burst they stall the wave at issue,
    // idling its matrix core. Load k of wave w is instruction 4k + w of its area
    // (input rows k < KX, halo rows KX <= k < KX + 2, dy rows after), so every
    // load's area and staged row are known at compile time up to the wave's bits.
    // A lane whose voxel lies outside the tile or the output, or a unit past the
    // last, loads zeros (out-of-range offset).
    static_assert(kLoader || (C::X_INSTR % 4 == 0 && C::Y_INSTR % 4 == 0 && C::XH_INSTR <= 8), "load slots");
    static_assert(C::XRY % (4 / C::IPR_X) == 0 && BY % (4 / C::IPR_Y) == 0, "a slot's rows share a plane");
    constexpr int KX = C::X_INSTR / 4, KH0 = KX, KY0 = KX + 2;
    constexpr int KLOADS = KY0 + C::Y_INSTR / 4;
    constexpr int RKX = 4 / C::IPR_X, RKY = 4 / C::IPR_Y;  // staged rows per slot
    const int wrx = wave / C::IPR_X, pcx = wave % C::IPR_X;
    const int wry = wave / C::IPR_Y, pcy = wave % C::IPR_Y;
    const uint32_t lxw = lxm + uint32_t(pcx * XPI * C::CIN * 2);
    const uint32_t lyw = lym + uint32_t(pcy * YPI * C::COUT * 2);
    __amdgpu_buffer_rsrc_t st_rx = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.tile), short(0),
                                                                     int(a.tile_bytes), 0x00020000);
    __amdgpu_buffer_rsrc_t st_ry = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.dy), short(0),
                                                                     int(a.dy_bytes), 0x00020000);
    __amdgpu_buffer_rsrc_t st_rl = st_rx, st_rh = st_rx;
    bool st_touch = false;
    char* st_dst = lds;
    uint32_t st_xorg = 0, st_yorg = 0;
    int32_t st_i0 = 0, st_i1 = 0, st_i2 = 0, st_o0 = 0, st_o1 = 0;
    bool st_live = false, st_okx = false, st_oky = false;
    auto stage_setup = [&](const Pos& p, int buf) {
        st_live = p.brick < a.nbricks;
        const uint32_t nn = st_live ? p.nn : 0;
        st_o0 = st_live ? p.bz * BZ : 0;
        st_o1 = st_live ? p.by * BY : 0;
        const int o2 = p.j * 32;
        st_i0 = st_o0 - a.pad[0];
        st_i1 = st_o1 - a.pad[1];
        st_i2 = o2 - a.pad[2];
        st_xorg = uint32_t(st_i0) * a.xplane + uint32_t(st_i1 + wrx) * a.xrow + uint32_t(st_i2) * (C::CIN * 2);
        st_yorg = uint32_t(st_o0) * a.yplane + uint32_t(st_o1 + wry) * a.yrow + uint32_t(o2) * (C::COUT * 2);
        st_okx = st_live && uint32_t(st_i2 + pcx * XPI + vx) < uint32_t(a.P[2]);
        st_oky = st_live && o2 + pcy * YPI + vy < a.O[2];
        st_rx = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.tile) + int64_t(nn) * a.tile_bytes, short(0),
                                                  int(a.tile_bytes), 0x00020000);
        st_ry = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.dy) + int64_t(nn) * a.dy_bytes, short(0),
                                                  int(a.dy_bytes), 0x00020000);
        if (FOLD) {
            st_rl = slab_rsrc(0, nn);
            st_rh = slab_rsrc(1, nn);
            st_touch = touches(st_i0, st_i1);
        }
        st_dst = lds + buf * C::STAGE_BYTES + wave * 1024;
    };
    auto stage_load = [&](int k) {
        if (k < KH0) {
            const int zr = (RKX * k) / C::XRY, yr0 = (RKX * k) % C::XRY;
            const bool ok = st_okx && uint32_t(st_i0 + zr) < uint32_t(a.P[0]) &&
                            uint32_t(st_i1 + yr0 + wrx) < uint32_t(a.P[1]);
            const uint32_t u = st_xorg + uint32_t(zr) * a.xplane + uint32_t(yr0) * a.xrow + lxw;
            xload(st_rx, st_rl, st_rh, st_dst + 4 * k * 1024, u, ok, st_i0 + zr, st_i1 + yr0 + wrx, st_touch);
        } else if (k < KY0) {
            const int hi = 4 * (k - KH0) + wave;
            if (hi < C::XH_INSTR) {
                const int row = hi * HRPI + hrow;
                const int zr = row / C::XRY, yr = row % C::XRY;
                const bool ok = st_live && uint32_t(st_i0 + zr) < uint32_t(a.P[0]) &&
                                uint32_t(st_i1 + yr) < uint32_t(a.P[1]) && uint32_t(st_i2 + hv) < uint32_t(a.P[2]);
                const uint32_t u = st_xorg - uint32_t(wrx) * a.xrow + uint32_t(zr) * a.xplane +
                                   uint32_t(yr) * a.xrow + lxh;
                xload(st_rx, st_rl, st_rh, st_dst + C::X_BYTES + 4 * (k - KH0) * 1024, u, ok, st_i0 + zr, st_i1 + yr,
                      st_touch);
            }
        } else {
            const int kk = k - KY0;
            const int zb = (RKY * kk) / BY, yb0 = (RKY * kk) % BY;
            const bool ok = st_oky && st_o0 + zb < a.O[0] && st_o1 + yb0 + wry < a.O[1];
            const uint32_t u = st_yorg + uint32_t(zb) * a.yplane + uint32_t(yb0) * a.yrow + lyw;
            // dy is read once per brick: nontemporal (cache policy NT)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(st_ry,
                                                     SC_LDSW(st_dst + C::X_BYTES + C::XH_BYTES + 4 * kk * 1024), 16,
                                                     ok ? u : a.dy_bytes, 0, 0, 2);
        }
    };
    // rows of a tile over which the loads of the next unit are spread (the rest
    // of the tile covers their latency)
    constexpr int LOAD_ROWS = C::NQ > 4 ? C::NQ - 2 : 1;
    static_assert(kLoader || (KLOADS + LOAD_ROWS - 1) / LOAD_ROWS <= 6, "at most one load per MFMA group");

    // the dedicated loaders issue every load of a unit: loader LI of KS issues the
    // instructions i with i % KS == LI (instruction index known at compile time)
    auto loader_unit = [&](const Pos& p, int buf, auto li_c) {
        constexpr int LI = decltype(li_c)::value;
        const bool live = p.brick < a.nbricks;
        const uint32_t nn = live ? p.nn : 0;
        const int o0 = live ? p.bz * BZ : 0, o1 = live ? p.by * BY : 0, o2 = p.j * 32;
        const int i0 = o0 - a.pad[0], i1 = o1 - a.pad[1], i2 = o2 - a.pad[2];
        const uint32_t xorg = uint32_t(i0) * a.xplane + uint32_t(i1) * a.xrow + uint32_t(i2) * (C::CIN * 2);
        const uint32_t yorg = uint32_t(o0) * a.yplane + uint32_t(o1) * a.yrow + uint32_t(o2) * (C::COUT * 2);
        __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.tile) + int64_t(nn) * a.tile_bytes, short(0), int(a.tile_bytes), 0x00020000);
        __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.dy) + int64_t(nn) * a.dy_bytes, short(0), int(a.dy_bytes), 0x00020000);
        const __amdgpu_buffer_rsrc_t rl = FOLD ? slab_rsrc(0, nn) : rx, rh = FOLD ? slab_rsrc(1, nn) : rx;
        const bool touch = touches(i0, i1);
        char* dst = lds + buf * C::STAGE_BYTES;
#pragma unroll
        for (int i = LI; i < C::X_INSTR; i += KS) {
            const int row = i / C::IPR_X, pc = i % C::IPR_X;
            const int zr = row / C::XRY, yr = row % C::XRY;
            const bool ok = live & (uint32_t(i0 + zr) < uint32_t(a.P[0])) & (uint32_t(i1 + yr) < uint32_t(a.P[1])) &
                            (uint32_t(i2 + pc * XPI + vx) < uint32_t(a.P[2]));
            const uint32_t u = xorg + uint32_t(zr) * a.xplane + uint32_t(yr) * a.xrow + lxm +
                               uint32_t(pc * XPI * C::CIN * 2);
            xload(rx, rl, rh, dst + i * 1024, u, ok, i0 + zr, i1 + yr, touch);
        }
#pragma unroll
        for (int hi = LI; hi < C::XH_INSTR; hi += KS) {
            const int row = hi * HRPI + hrow;
            const int zr = row / C::XRY, yr = row % C::XRY;
            const bool ok = live & (uint32_t(i0 + zr) < uint32_t(a.P[0])) & (uint32_t(i1 + yr) < uint32_t(a.P[1])) &
                            (uint32_t(i2 + hv) < uint32_t(a.P[2]));
            const uint32_t u = xorg + uint32_t(zr) * a.xplane + uint32_t(yr) * a.xrow + lxh;
            xload(rx, rl, rh, dst + C::X_BYTES + hi * 1024, u, ok, i0 + zr, i1 + yr, touch);
        }
#pragma unroll
        for (int j = LI; j < C::Y_INSTR; j += KS) {
            const int row = j / C::IPR_Y, pc = j % C::IPR_Y;
            const int zb = row / BY, yb = row % BY;
            const bool ok = live & (o0 + zb < a.O[0]) & (o1 + yb < a.O[1]) & (o2 + pc * YPI + vy < a.O[2]);
            const uint32_t u = yorg + uint32_t(zb) * a.yplane + uint32_t(yb) * a.yrow + lym +
                               uint32_t(pc * YPI * C::COUT * 2);
            // dy is read once per brick: nontemporal (cache policy NT; the C3
            // weight gradient 1-1.5 % faster than with cached loads)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ry, SC_LDSW(dst + C::X_BYTES + C::XH_BYTES + j * 1024), 16,
                                                     ok ? u : a.dy_bytes, 0, 0, 2);
        }
    };
    if (KS == 2 && simd == 3) {
        auto run_loader = [&](auto li_c) {
            Pos sp{L, 0, 0, 0, 0, 0};
            seg_start(sp);
            uint32_t u = 0;
            int b = 0;
            while (sp.brick < a.nbricks) {
                if (u >= uint32_t(NB)) spin_until(flag_free0 + uint32_t(4 * b), uint32_t(NCW) * (u / NB));
                loader_unit(sp, b, li_c);
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                raise(flag_full0 + uint32_t(4 * b));
                advance(sp);
                ++u;
                b = b + 1 == NB ? 0 : b + 1;
            }
        };
        if (ks == 0)
            run_loader(std::integral_constant<int, 0>{});
        else
            run_loader(std::integral_constant<int, KS - 1>{});
        return;
    }
    if (KS == 1 && kLoader && simd == 3) {
        auto run_loader = [&](auto li_c) {
            Pos cp{L, 0, 0, 0, 0, 0}, sp{L, 0, 0, 0, 0, 0};
            seg_start(cp);
            seg_start(sp);
            loader_unit(sp, 0, li_c);
            advance(sp);
            int buf = 0;
            while (cp.brick < a.nbricks) {
                // this tile's loads have landed and the compute waves are done
                // with the other buffer: fill it with the next unit
                wait_vm_barrier<0>();
                loader_unit(sp, buf ^ 1, li_c);
                advance(sp);
                buf ^= 1;
                advance(cp);
            }
            wait_vm_barrier<0>();
        };
        run_loader(std::integral_constant<int, 0>{});
        return;
    }

    // ---- operand reads (compute waves) ----
    // transposed-read lane terms: 16-lane group G = lane / 16 reads voxels
    // 16g + 4r + i/4 (g = lane / 32, read r) at channels c0 + 4 (i % 4) .. + 3,
    // c0 = 32 * tile + 16 * (G % 2)
    const int gi = lane & 15, gh = lane >> 5, gc = (lane >> 4) & 1;
    const int vq = 16 * gh + gi / 4;  // voxel of read 0
    auto lane_off = [&](int upv, int c) {
        const int swz = upv == 8 ? (((vq >> 1) & 1) << 1) : 0;
        return uint32_t(vq * upv * 16 + (((c >> 3) ^ swz) << 4) + (c & 7) * 2);
    };
    const uint32_t xl = lane_off(C::UPX, 32 * cb + 16 * gc + 4 * (gi & 3));
    const uint32_t yl = lane_off(C::UPY, 32 * mb + 16 * gc + 4 * (gi & 3));

    // K steps of 16 voxels per wave and row (both, or the wave's half), and the
    // transposed reads they need: K step s of lane half g multiplies voxels
    // 16g + 8s .. + 7 and, shifted by kw <= 2, needs voxels up to 16g + 8s + 9,
    // which reads 2s .. 2s + 2 cover (read 4 of lane half 1 is the halo area).
    constexpr int SW = 2 / KS;
    constexpr int NXR = 2 * SW + 1, NYR = 2 * SW;
    const int s0 = KS == 2 ? ks : 0;

    f32x16_w acc[3][3];
#pragma unroll
    for (int kh = 0; kh < 3; ++kh)
#pragma unroll
        for (int kw = 0; kw < 3; ++kw)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[kh][kw][e] = 0.f;

    // register slots: input rows of plane parity p, row yr in slot p * 4 + yr % 4
    uint32_t xr[8][2 * NXR];
    uint32_t xs[8][4 * SW];     // kw = 1 windows (the wave's K steps) of the slot's row
    uint32_t dyr[2][4 * SW];    // dy of output rows q (parity q % 2), the wave's K steps

    // read 4 (voxels 16g + 16 .. + 19): lane half 0 from the main row, lane half 1
    // (voxels 32..35) from the halo area
    const int vq4 = gh ? gi / 4 : 16 + gi / 4;
    const uint32_t xl4 = uint32_t(gh ? C::X_BYTES : 0) +
                         uint32_t(vq4 * C::UPX * 16 +
                                  ((((32 * cb + 16 * gc + 4 * (gi & 3)) >> 3) ^ wx_swz<C::UPX>(vq4)) << 4) +
                                  ((4 * (gi & 3)) & 7) * 2);
    const uint32_t xrs4 = uint32_t(gh ? C::XH_ROW : C::XROW);
    // reads j < NXR - 1 are main-row reads 2 s0 + j; the last one is read
    // 2 s0 + NXR - 1, which is read 4 (halo form) unless it is the first half's read 2
    constexpr uint32_t RSTEP_X = 4 * C::UPX * 16, RSTEP_Y = 4 * C::UPY * 16;
    const uint32_t xl_s = xl + uint32_t(2 * s0) * RSTEP_X;
    const bool last_halo = 2 * s0 + NXR - 1 == 4;
    const uint32_t xl_last = last_halo ? xl4 : xl_s + uint32_t(NXR - 1) * RSTEP_X;
    const uint32_t xst_last = last_halo ? xrs4 : uint32_t(C::XROW);
    const uint32_t yl_s = yl + uint32_t(2 * s0) * RSTEP_Y;
    auto read_x_row = [&](uint32_t xbase, int zr, int yr, int slot) {
        const int row = zr * C::XRY + yr;
        const uint32_t base = xbase + uint32_t(row * C::XROW) + xl_s;
#pragma unroll
        for (int j = 0; j < NXR - 1; ++j) {
            const uint2 d = lds_read_tr16_b64(base + uint32_t(j) * RSTEP_X);
            xr[slot][2 * j] = d.x;
            xr[slot][2 * j + 1] = d.y;
        }
        const uint2 d = lds_read_tr16_b64(xbase + xl_last + uint32_t(row) * xst_last);
        xr[slot][2 * NXR - 2] = d.x;
        xr[slot][2 * NXR - 1] = d.y;
    };
    auto read_dy_row = [&](uint32_t ybase, int q, int slot) {
        const uint32_t base = ybase + uint32_t(q * C::YROW) + yl_s;
#pragma unroll
        for (int j = 0; j < NYR; ++j) {
            const uint2 d = lds_read_tr16_b64(base + uint32_t(j) * RSTEP_Y);
            dyr[slot][2 * j] = d.x;
            dyr[slot][2 * j + 1] = d.y;
        }
    };
    // reads for output row q: its dy row and the input rows it needs first
    auto issue_row = [&](uint32_t xbase, uint32_t ybase, int q) {
        const int zb = q / BY, yb = q % BY;
        read_dy_row(ybase, q, q & 1);
        if (yb == 0) {
#pragma unroll
            for (int kh = 0; kh < 3; ++kh) read_x_row(xbase, zb + kd, kh, (zb & 1) * 4 + kh);
        } else {
            read_x_row(xbase, zb + kd, yb + 2, (zb & 1) * 4 + (yb + 2) % 4);
        }
    };
    auto ready_row = [&](int q) {
        const int zb = q / BY, yb = q % BY;
#pragma unroll
        for (int e = 0; e < 4 * SW; ++e) lds_ready(dyr[q & 1][e]);
        const int k0 = yb == 0 ? 0 : 2;
#pragma unroll
        for (int kh = k0; kh < 3; ++kh) {
            const int slot = (zb & 1) * 4 + (yb + kh) % 4;
#pragma unroll
            for (int e = 0; e < 2 * NXR; ++e) lds_ready(xr[slot][e]);
            // kw = 1: voxels shifted by one (the high half of dword i, the low of i + 1)
#pragma unroll
            for (int sl = 0; sl < SW; ++sl)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    xs[slot][4 * sl + e] =
                        __builtin_amdgcn_alignbit(xr[slot][4 * sl + e + 1], xr[slot][4 * sl + e], 16);
        }
    };
    // after_group(g) runs after MFMA group g = sl * 3 + kh (three MFMAs) of the row
    auto mfma_row = [&](int q, auto&& after_group) {
        const int zb = q / BY, yb = q % BY;
#pragma unroll
        for (int sl = 0; sl < SW; ++sl) {
            const uint4 av = make_uint4(dyr[q & 1][4 * sl], dyr[q & 1][4 * sl + 1], dyr[q & 1][4 * sl + 2],
                                        dyr[q & 1][4 * sl + 3]);
#pragma unroll
            for (int kh = 0; kh < 3; ++kh) {
                const int slot = (zb & 1) * 4 + (yb + kh) % 4;
                const uint32_t* x = xr[slot];
                const uint4 b0 = make_uint4(x[4 * sl], x[4 * sl + 1], x[4 * sl + 2], x[4 * sl + 3]);
                const uint4 b1 = make_uint4(xs[slot][4 * sl], xs[slot][4 * sl + 1], xs[slot][4 * sl + 2],
                                            xs[slot][4 * sl + 3]);
                const uint4 b2 = make_uint4(x[4 * sl + 1], x[4 * sl + 2], x[4 * sl + 3], x[4 * sl + 4]);
                acc[kh][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                                     __builtin_bit_cast(bf16x8_w, b0), acc[kh][0], 0,
                                                                     0, 0);
                acc[kh][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                                     __builtin_bit_cast(bf16x8_w, b1), acc[kh][1], 0,
                                                                     0, 0);
                acc[kh][2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_w, av),
                                                                     __builtin_bit_cast(bf16x8_w, b2), acc[kh][2], 0,
                                                                     0, 0);
                after_group(sl * 3 + kh);
            }
        }
    };

    Pos cp{L, 0, 0, 0, 0, 0}, sp{L, 0, 0, 0, 0, 0};
    seg_start(cp);
    seg_start(sp);
    if (!kLoader) {
        stage_setup(sp, 0);
#pragma unroll
        for (int k = 0; k < KLOADS; ++k) stage_load(k);
        advance(sp);
    }
    int buf = 0;
    uint32_t u = 0;
    while (cp.brick < a.nbricks) {
        // this tile's loads have landed (and, with barriers, every wave is done
        // with the buffer that is refilled next)
        if (KS == 2)
            spin_until(flag_full0 + uint32_t(4 * buf), 2u * (u / NB + 1));
        else
            wait_vm_barrier<0>();
        const uint32_t xbase = lds0 + uint32_t(buf * C::STAGE_BYTES);
        const uint32_t ybase = xbase + uint32_t(C::X_BYTES + C::XH_BYTES);
        if (!kLoader) {
            stage_setup(sp, buf ^ 1);
            advance(sp);
        }
        issue_row(xbase, ybase, 0);
#pragma unroll
        for (int q = 0; q < C::NQ; ++q) {
            const bool plane_break = (q + 1) % BY == 0;  // next row starts a new plane
            if (q + 1 < C::NQ && !plane_break) {
                issue_row(xbase, ybase, q + 1);
                lds_wait<NXR + NYR>();
            } else {
                lds_wait<0>();
            }
            ready_row(q);
            // the next unit's loads go out one per MFMA group, so that the memory
            // pipeline never holds more than about one load per wave
            const int kb = !kLoader && q < LOAD_ROWS ? (q * KLOADS + LOAD_ROWS - 1) / LOAD_ROWS : KLOADS;
            const int ke = !kLoader && q < LOAD_ROWS ? ((q + 1) * KLOADS + LOAD_ROWS - 1) / LOAD_ROWS : KLOADS;
            mfma_row(q, [&](int g) {
                if (kb + g < ke) stage_load(kb + g);
            });
            if (q + 1 < C::NQ && plane_break) issue_row(xbase, ybase, q + 1);
        }
        // the last row waited for all of this wave's reads of the buffer
        if (KS == 2) raise(flag_free0 + uint32_t(4 * buf));
        buf = buf + 1 == NB ? 0 : buf + 1;
        ++u;
        advance(cp);
    }
    if (KS == 1) wait_vm_barrier<0>();
    {
        // partial: [workgroup][K half][role][tap kh * 3 + kw][lane][16]
        float4* out = reinterpret_cast<float4*>(a.part + (int64_t(L) * KS + s0) * C::PART_FLOATS +
                                                int64_t(role) * 9 * 1024);
#pragma unroll
        for (int kh = 0; kh < 3; ++kh)
#pragma unroll
            for (int kw = 0; kw < 3; ++kw)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4)
                    out[((kh * 3 + kw) * 64 + lane) * 4 + r4] =
                        make_float4(acc[kh][kw][4 * r4], acc[kh][kw][4 * r4 + 1], acc[kh][kw][4 * r4 + 2],
                                    acc[kh][kw][4 * r4 + 3]);
    }
}

// The partials are summed in two fixed-order passes: pass 1 gives each of
// kChunks blocks of workgroup partials its own sum (one thread per partial float
// and chunk, many independent chains instead of one chain of nsplit loads),
// pass 2 adds the kChunks sums in order and scatters into dw. Bitwise
// repeatable.
constexpr int kChunks = 16;

template <int KD, int NCI, int NCO>
__global__ __launch_bounds__(256) void wgrad_xm_reduce1(const float* part, float* sums, int nsplit)
{
    constexpr int NR = NCO * NCI * KD;
    constexpr int BLK = 4 * 9 * 1024;
    constexpr int NE = NR * 9 * 1024;
    const int e = int(blockIdx.x) * 256 + threadIdx.x;
    const int ch = int(blockIdx.y);
    if (e >= NE) return;
    const int per = (nsplit + kChunks - 1) / kChunks;
    const int s0 = ch * per, s1 = min(nsplit, s0 + per);
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
    int sp = s0;
    for (; sp + 4 <= s1; sp += 4) {
#pragma unroll
        for (int j = 0; j < 4; ++j) s4[j] += part[int64_t(sp + j) * BLK + e];
    }
    for (int j = 0; sp + j < s1; ++j) s4[j] += part[int64_t(sp + j) * BLK + e];
    sums[int64_t(ch) * NE + e] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
}

// dw[co][ci][tap] = sum over the chunk sums, in chunk order; NaN everywhere when
// the partial kernel reported a hand-off wait that gave up.
template <int KD, int NCI, int NCO>
__global__ __launch_bounds__(256) void wgrad_xm_reduce2(const float* sums, float* dw, const uint32_t* status)
{
    constexpr int NR = NCO * NCI * KD;
    constexpr int CIN = 32 * NCI;
    constexpr int TAPS = KD * 9;
    constexpr int NE = NR * 9 * 1024;
    const int e = int(blockIdx.x) * 256 + threadIdx.x;
    if (e >= NE) return;
    const int r = e % 16, lane = (e / 16) % 64, t9 = (e / 1024) % 9, wave = e / (9 * 1024);
    const int kd = wave % KD, cb = (wave / KD) % NCI, mb = wave / (KD * NCI);
    const int co = mb * 32 + 8 * (r / 4) + 4 * (lane / 32) + (r % 4);
    const int ci = cb * 32 + (lane % 32);
    const int tap = kd * 9 + t9;
    float acc = 0.f;
#pragma unroll
    for (int ch = 0; ch < kChunks; ++ch) acc += sums[int64_t(ch) * NE + e];
    dw[(co * CIN + ci) * TAPS + tap] = status[0] == 0u ? acc : __builtin_nanf("");
}

struct WxPlan {
    bool ok;
    int cfg;  // 0: KD 3, 32 -> 32 channels, brick 2 x 4, K split in halves (8 waves); 1: KD 1, 64 -> 64, brick 1 x 8
    int ks;   // K splits per workgroup (partials per workgroup)
    WxArgs a;
    size_t lds;
    int64_t grid;
};

// Brick and stage depth of the three-role (KD = 3, 32 -> 32 channels) kernel.
constexpr int kC3BZ = 2, kC3BY = 4, kC3NB = 2;

WxPlan plan_wx(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    WxPlan p{};
    p.ok = false;
    if (force_generic() || force_tiled() || dt != SHARD_BF16) return p;
    for (int k = 0; k < 3; ++k)
        if (cv.S[k] != 1 || std::abs(cv.pad[k]) > (1 << 20) || cv.O[k] >= (int64_t(1) << 24) ||
            t.P[k] >= (int64_t(1) << 24))
            return p;
    if (cv.K[1] != 3 || cv.K[2] != 3) return p;
    int bz, by;
    if (cv.K[0] == 3 && t.c == 32 && cv.cout == 32) {
        p.cfg = 0;
        p.ks = 2;
        bz = kC3BZ, by = kC3BY;
        p.lds = 0;
    } else if (cv.K[0] == 1 && t.c == 64 && cv.cout == 64) {
        p.cfg = 1;
        p.ks = 1;
        bz = 1, by = 8;
        p.lds = WxCfg<1, 2, 2, 1, 8>::LDS_BYTES;
    } else {
        return p;
    }
    const int64_t tb = t.P[0] * t.P[1] * t.P[2] * t.c * 2;
    const int64_t db = cv.O[0] * cv.O[1] * cv.O[2] * cv.cout * 2;
    if (tb >= (int64_t(1) << 32) - 64 || db >= (int64_t(1) << 32) - 64) return p;
    WxArgs& a = p.a;
    for (int k = 0; k < 3; ++k) {
        a.P[k] = int32_t(t.P[k]);
        a.O[k] = int32_t(cv.O[k]);
        a.pad[k] = int32_t(cv.pad[k]);
    }
    a.NBZ = int32_t(ceil_div(cv.O[0], bz));
    a.NBY = int32_t(ceil_div(cv.O[1], by));
    pick_raster(a.NBZ, a.NBY, 8, a.TZ, a.TY);
    a.NXT = int32_t(ceil_div(cv.O[2], 32));
    const int64_t rows = t.n * int64_t(a.NBZ) * a.NBY;
    if (rows == 0 || a.NXT == 0) return p;
    int64_t nseg, T;
    pick_segments(rows, a.NXT, 256, 0, 4, nseg, T);
    a.nseg = int32_t(nseg);
    a.T = int32_t(T);
    const int64_t nb = rows * nseg;
    if (nb >= (int64_t(1) << 31)) return p;
    a.nbricks = uint32_t(nb);
    a.tile_bytes = uint32_t(tb);
    a.dy_bytes = uint32_t(db);
    a.xrow = uint32_t(t.P[2] * t.c * 2);
    a.xplane = uint32_t(t.P[1] * t.P[2] * t.c * 2);
    a.yrow = uint32_t(cv.O[2] * cv.cout * 2);
    a.yplane = uint32_t(cv.O[1] * cv.O[2] * cv.cout * 2);
    p.grid = std::max<int64_t>(1, std::min<int64_t>(nb, 256));
    p.ok = true;
    return p;
}

template <int KD, int NCI, int NCO, int BZ, int BY, int KS, int NB>
hipError_t run_wx(const WxPlan& p, float* dw, bool fold, uint32_t* status, hipStream_t s)
{
    using C = WxCfg<KD, NCI, NCO, BZ, BY>;
    constexpr int LDS = NB * C::STAGE_BYTES + (KS == 2 ? 8 * NB + 16 : 0);
    static_assert(LDS <= 160 * 1024, "LDS budget");
    auto fn = fold ? &wgrad_xm<KD, NCI, NCO, BZ, BY, KS, NB, true> : &wgrad_xm<KD, NCI, NCO, BZ, BY, KS, NB, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       LDS);
    if (e != hipSuccess) return e;
    WxArgs a = p.a;
    void* args[] = {&a};
    e = hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(p.grid)), dim3(256 * KS), args, LDS, s);
    if (e != hipSuccess) return e;
    const int total = C::NR * 9 * 1024;
    float* sums = p.a.part + size_t(p.grid) * KS * C::PART_FLOATS;
    hipLaunchKernelGGL((wgrad_xm_reduce1<KD, NCI, NCO>), dim3(unsigned(ceil_div(total, 256)), kChunks), dim3(256), 0,
                       s, p.a.part, sums, int(p.grid * KS));
    hipLaunchKernelGGL((wgrad_xm_reduce2<KD, NCI, NCO>), dim3(unsigned(ceil_div(total, 256))), dim3(256), 0, s, sums,
                       dw, static_cast<const uint32_t*>(status));
    return hipGetLastError();
}

}  // namespace

size_t wgrad_xm_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    const WxPlan p = plan_wx(t, cv, dt);
    // partials, then kChunks chunk sums of at most four roles
    return p.ok ? (size_t(p.grid) * size_t(p.ks) + kChunks) * 4 * 9 * 1024 * sizeof(float) : 0;
}

// The W-march weight gradient applies to bf16, unit stride, 3 x 3 taps in H and
// W with 3 (Ci = Co = 32) or 1 (Ci = Co = 64) taps in D, tiles and dy of < 4 GiB
// per batch item, 16-byte aligned buffers. Launches the partial and the reduce
// kernels; returns hipErrorNotSupported when it does not apply.
// With a folded halo the margins must lie on one axis, 0 or 1, the slabs be
// 16-byte aligned and below 4 GiB per batch item.
hipError_t launch_wgrad_xm(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* dw, void* ws, const Fold* fold, uint32_t* status, hipStream_t s)
{
    WxPlan p = plan_wx(t, cv, dt);
    if (!p.ok || reinterpret_cast<uintptr_t>(tile) % 16 != 0 || reinterpret_cast<uintptr_t>(dy) % 16 != 0 ||
        reinterpret_cast<uintptr_t>(ws) % 16 != 0)
        return hipErrorNotSupported;
    p.a.fa = -1;
    if (fold) {
        if (fold->mask != 1u && fold->mask != 2u) return hipErrorNotSupported;
        const int k = fold->mask == 1u ? 0 : 1;
        p.a.fa = k;
        p.a.flo = int32_t(t.lo[k]);
        p.a.fhi = int32_t(t.lo[k] + t.ext[k]);
        for (int sd = 0; sd < 2; ++sd) {
            const int64_t w = sd == 0 ? t.lo[k] : t.hi[k];
            const char* sp = fold->slab[k][sd];
            if (reinterpret_cast<uintptr_t>(sp) % 16 != 0) return hipErrorNotSupported;
            // slab [P0 or w][w or P1][P2][c]: no margins on the other axes
            const int64_t sz = k == 0 ? int64_t(p.a.xplane) : w * int64_t(p.a.xrow);
            const int64_t bb = (k == 0 ? w : t.P[0]) * sz;
            if (bb >= (int64_t(1) << 32) - 64) return hipErrorNotSupported;
            p.a.fslab[sd] = w > 0 ? sp : nullptr;
            p.a.fbatch[sd] = uint32_t(bb);
            p.a.fSZ[sd] = uint32_t(sz);
        }
    }
    p.a.tile = static_cast<const char*>(tile);
    p.a.dy = static_cast<const char*>(dy);
    p.a.part = static_cast<float*>(ws);
    p.a.status = status;
    p.a.wait_polls = call_opts().wait_polls ? call_opts().wait_polls : kDefaultWaitPolls;
    return p.cfg == 0 ? run_wx<3, 1, 1, kC3BZ, kC3BY, 2, kC3NB>(p, dw, fold != nullptr, status, s)
                      : run_wx<1, 2, 2, 1, 8, 1, 2>(p, dw, fold != nullptr, status, s);
}

}  // namespace shardconv
