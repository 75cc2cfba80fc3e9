// Forward convolution, bf16, unit stride, kernel width 3 along the innermost
// axis (the halo-padded 3D/2D shard workloads): a persistent implicit GEMM with
// M = 32 input voxels of one W row, N = 32 output channels, K = 16 input
// channels per v_mfma_f32_32x32x16_bf16.
//
//  * The weights of a wave's 32 output channels sit in registers (B fragments)
//    for the kernel's lifetime, so LDS carries input rows only.
//  * A workgroup (4 waves) owns a brick of BZ x BY output rows and marches along
//    W in 32-voxel input tiles. Each tile's footprint (BZ+KD-1 x BY+KH-1 input
//    rows of 32 voxels, all channels) is staged by direct global->LDS buffer
//    loads, NBUF deep; voxels outside the tile load as zero (out-of-range buffer
//    offsets), which is the zero padding.
//  * Taps along H/D are row choices: input row j of the stage serves the wave's
//    output rows j - kh. Taps along W are not applied to the operand at all: input
//    voxel u reaches output u - kw through tap kw, so each (output row, kw) keeps
//    its own accumulator over the same A fragments and the three are summed with a
//    shift of kw rows when the tile is done. Tile j stages tile voxels
//    [32j, 32j + 32); output rows that straddle the tile edge take their missing
//    terms from the previous tile (a 3-value carry, zero before the row's first
//    tile), so tile j completes the outputs [32j + pad - 2, 32j + pad + 30). A row
//    takes ceil(P2 / 32) tiles: the last two outputs of the last tile need only
//    voxels past the row end (zero), so they are written from the carry (no
//    extra tile of MFMAs for them).
//  * A-row m of the MFMA holds input voxel x(m) = 16*((m>>2)&1) + 4*(m>>3) + (m&3),
//    so that accumulator register r of lane half g is voxel 16g + r: the W shift is
//    a register shift except at r < kw, where the value comes from the other lane
//    half (one ds_bpermute per value) or from the carry.
//  * Staged rows are [x][16-byte unit], the unit XOR-swizzled by bits of x so the
//    16 lanes of each ds_read_b128 phase hit distinct bank groups.
//  * Results leave through a per-wave LDS transpose as 16-byte buffer stores;
//    stores of outputs outside the tensor get an out-of-range offset and are
//    dropped, so every wave issues the same number of memory operations per tile
//    and the vmcnt waits are compile-time constants (vector memory operations
//    complete in issue order).
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_r;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_r;
typedef __attribute__((ext_vector_type(16))) float f32x16_r;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_r;

#define SC_LDS(p) ((__attribute__((address_space(3))) void*)(p))

namespace {

struct XmArgs {
    const char* tile;
    const char* wfrag;
    char* y;
    int32_t P[3], O[3];
    int32_t pad[3];
    int32_t NBZ, NBY, NXT;  // bricks along D and H, input tiles along W
    int32_t TZ, TY;         // raster block of TZ x TY bricks (divides NBZ x NBY)
    int32_t nseg, T;        // W segments per row and their length in tiles
    uint32_t nbricks;       // n * NBZ * NBY * nseg
    uint32_t batch_bytes;   // tile bytes per batch item (< 2^32)
    uint32_t ybatch_bytes;  // output bytes per batch item (< 2^32)
    int32_t cout;
    int32_t org[2], oend[2];  // computed outputs along axes 0, 1: [org, oend) (O gives the strides)
    // a second region along axis 0 in the same launch: bricks bz >= nbz_a cover
    // axis-0 rows [org0b, oend0b) (same axes 1 and 2)
    int32_t nbz_a, org0b, oend0b;
    // halo folded into the loads along axis fa (0 or 1): padded rows c < flo come
    // from fslab[0], rows c >= fhi from fslab[1] (null: zero), the rest from the tile
    const char* fslab[2];
    uint32_t fbatch[2];  // slab bytes per batch item
    uint32_t fSZ[2];     // slab stride along axis 0, bytes
    int32_t fa, flo, fhi;
};

// 16-byte unit swizzle of voxel x for UPV units per voxel (see file comment).
template <int UPV>
__device__ __forceinline__ constexpr int xm_swz(int x)
{
    return UPV == 4 ? (((x >> 2) & 1) | (((x >> 4) & 1) << 1))
                    : (((x >> 1) & 1) | (((x >> 2) & 1) << 1) | (((x >> 4) & 1) << 2));
}

template <int CIN, int KD, int KH, int WZ, int WY, int WC, int R, int NBUF>
struct XmCfg {
    static_assert(CIN == 32 || CIN == 64, "16-byte units per voxel: 4 or 8");
    static_assert(WZ * WY * WC == 4, "four waves");
    static_assert(NBUF >= 2 && NBUF <= 4, "stage depth");
    // a tile's last row is finished while the next tile's first row multiplies:
    // they need distinct accumulators
    static_assert(R >= 2, "two or more output rows per wave");
    static constexpr int KW = 3;
    static constexpr int UPV = CIN / 8;
    static constexpr int NKC = CIN / 16;
    static constexpr int BZ = WZ, BY = WY * R;
    static constexpr int IRZ = BZ + KD - 1, IRY = BY + KH - 1, IR = IRZ * IRY;
    static constexpr int ROW_BYTES = 32 * UPV * 16;
    static constexpr int STAGE_BYTES = IR * ROW_BYTES;
    static constexpr int RPI = 256 / (32 * UPV);  // staged rows per direct-load instruction
    static_assert(IRY % RPI == 0, "an instruction's rows share their D row");
    static constexpr int NIT = IR / RPI;          // direct loads per thread per stage
    static constexpr int NROWS_IN = R + KH - 1;
    static_assert(NROWS_IN < 16, "lgkmcnt range");
    static constexpr int EPI_BYTES = 2048;  // one 32 x 32 bf16 output tile per wave
    static constexpr int EPI_STORES = R * 2;
    static constexpr int LDS_BYTES = NBUF * STAGE_BYTES + 4 * EPI_BYTES;
    static constexpr int VM_BASE = NIT * (NBUF - 2);
    static_assert(NBUF <= 4 && VM_BASE + EPI_STORES * 2 < 64, "vmcnt range");
};

template <int CIN, int KD, int KH, int WZ, int WY, int WC, int R, int NBUF, bool FOLD>
__global__ __launch_bounds__(256, 1) void conv_fwd_xm(XmArgs a)
{
    using C = XmCfg<CIN, KD, KH, WZ, WY, WC, R, NBUF>;
    constexpr int KW = C::KW;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wc = wave % WC, wy = (wave / WC) % WY, wz = wave / (WC * WY);
    const int g = lane >> 5;
    const uint32_t G = gridDim.x;
    const uint32_t L = uint32_t(xcd_remap(blockIdx.x, G));

    // weights of this wave's output-channel tile -> registers
    u32x4_r wv[KD][KH][KW][C::NKC];
    {
        const u32x4_r* wf = reinterpret_cast<const u32x4_r*>(a.wfrag);
#pragma unroll
        for (int kd = 0; kd < KD; ++kd)
#pragma unroll
            for (int kh = 0; kh < KH; ++kh)
#pragma unroll
                for (int kw = 0; kw < KW; ++kw)
#pragma unroll
                    for (int kc = 0; kc < C::NKC; ++kc) {
                        const int tap = (kd * KH + kh) * KW + kw;
                        wv[kd][kh][kw][kc] = wf[((tap * C::NKC + kc) * WC + wc) * 64 + lane];
                    }
    }

    // staging: instruction it of a thread loads 16-byte unit su of voxel xs of
    // staged row it * RPI + hs (rows D-major, then H)
    const int hs = tid / (32 * C::UPV), xs = (tid % (32 * C::UPV)) / C::UPV, su = tid % C::UPV;
    const uint32_t SY = uint32_t(a.P[2]) * (CIN * 2), SZ = uint32_t(a.P[1]) * SY;
    const uint32_t tb = uint32_t(hs) * SY + uint32_t(xs * CIN * 2 + (su ^ xm_swz<C::UPV>(xs)) * 16);

    // A-read lane offsets within a staged row, per 16-channel chunk
    const int m = lane & 31;
    const int xa = 16 * ((m >> 2) & 1) + 4 * (m >> 3) + (m & 3);
    const uint32_t lds0 = lds_addr(lds);
    uint32_t abase[C::NKC];
#pragma unroll
    for (int kc = 0; kc < C::NKC; ++kc)
        abase[kc] = lds0 + uint32_t((wz * C::IRY + wy * R) * C::ROW_BYTES + xa * C::UPV * 16 +
                                    (((2 * kc) | g) ^ xm_swz<C::UPV>(xa)) * 16);

    // bricks L, L + G, ... ; brick b is W segment b % nseg of output rows b / nseg.
    // A segment after the first starts one tile early (its outputs are not stored)
    // to build the carry.
    // The brick's rows (bz, by) and batch item nn are decoded once per brick.
    struct Pos {
        uint32_t brick;
        int32_t j, jend, jstore;
        int32_t bz, by;
        uint32_t nn;
    };
    auto seg_start = [&](Pos& p) {
        if (p.brick >= a.nbricks) return;
        uint32_t t = p.brick / uint32_t(a.nseg);
        const int32_t seg = int32_t(p.brick - t * uint32_t(a.nseg));
        p.jstore = seg * a.T;
        p.j = seg > 0 ? p.jstore - 1 : 0;
        p.jend = min(p.jstore + a.T, a.NXT);
        brick_rows(t, a.NBZ, a.NBY, a.TZ, a.TY, p.bz, p.by, p.nn);
    };
    auto advance = [&](Pos& p) {
        if (++p.j >= p.jend) {
            p.brick += G;
            seg_start(p);
        }
    };

    // Staging of one unit is split in a set-up (uniform values of the unit, once per
    // tile) and NIT single loads that the main loop spreads over its MFMA steps:
    // issued as a burst, the loads stall the wave at issue (the memory pipeline
    // accepts them more slowly than four waves issue them), and with one wave per
    // SIMD every stalled cycle is an idle matrix core. Offsets are 32-bit (a batch
    // item is < 4 GiB); a voxel outside the tile, or a unit past the last, gets an
    // out-of-range offset and loads as zero.
    // first output row along axis 0 of brick row bz, and the end of its region
    auto org0_of = [&](int bz) { return bz < a.nbz_a ? a.org[0] + bz * C::BZ : a.org0b + (bz - a.nbz_a) * C::BZ; };
    auto end0_of = [&](int bz) { return bz < a.nbz_a ? a.oend[0] : a.oend0b; };
    __amdgpu_buffer_rsrc_t st_r = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.tile), short(0),
                                                                    int(a.batch_bytes), 0x00020000);
    // folded halo: the received slabs of this batch item (a missing slab is a
    // zero-length buffer, so its rows load as zero)
    __amdgpu_buffer_rsrc_t st_rl = st_r, st_rh = st_r;
    char* st_dst = lds;
    uint32_t st_vbase = 0;
    int32_t st_i0 = 0, st_i1 = 0, st_vy = 0;
    bool st_okx = false;
    auto stage_setup = [&](const Pos& p, int buf) {
        const bool live = p.brick < a.nbricks;
        const int bz = live ? p.bz : 0, by = live ? p.by : 0;
        const uint32_t nn = live ? p.nn : 0;
        st_i0 = org0_of(bz) - a.pad[0];
        st_i1 = a.org[1] + by * C::BY - a.pad[1];
        const int i2 = p.j * 32;
        const int64_t origin = ((int64_t(st_i0) * a.P[1] + st_i1) * a.P[2] + i2) * (CIN * 2);
        st_r = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.tile) + int64_t(nn) * a.batch_bytes, short(0),
                                                 int(a.batch_bytes), 0x00020000);
        if (FOLD) {
            st_rl = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<char*>(a.fslab[0] ? a.fslab[0] + int64_t(nn) * a.fbatch[0] : a.tile), short(0),
                a.fslab[0] ? int(a.fbatch[0]) : 0, 0x00020000);
            st_rh = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<char*>(a.fslab[1] ? a.fslab[1] + int64_t(nn) * a.fbatch[1] : a.tile), short(0),
                a.fslab[1] ? int(a.fbatch[1]) : 0, 0x00020000);
        }
        st_dst = lds + buf * C::STAGE_BYTES + wave * 64 * 16;
        st_vbase = uint32_t(origin) + tb;
        st_vy = st_i1 + hs;
        st_okx = live && uint32_t(i2 + xs) < uint32_t(a.P[2]);
    };
    auto stage_load = [&](int it) {
        const int row0 = it * C::RPI;
        const int rz = row0 / C::IRY, ry = row0 % C::IRY;
        const bool ok = st_okx && uint32_t(st_i0 + rz) < uint32_t(a.P[0]) && uint32_t(st_vy + ry) < uint32_t(a.P[1]);
        uint32_t off = st_vbase + uint32_t(rz) * SZ + uint32_t(ry) * SY;
        if (FOLD) {
            // the row's coordinate along the fold axis is uniform over the
            // instruction (one D row per instruction; one H row when fa == 1)
            const int32_t z = st_i0 + rz;
            const int32_t c = a.fa == 0 ? z : st_i1 + ry;
            const uint32_t sfa = a.fa == 0 ? SZ : SY;
            // one load per branch: the buffer descriptor stays scalar (a select of
            // descriptors compiles to a per-lane loop)
            if (c < a.flo) {
                off -= uint32_t(z) * (SZ - a.fSZ[0]);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(st_rl, SC_LDS(st_dst + it * 4096), 16,
                                                         ok ? off : 0xFFFFFFC0u, 0, 0, 0);
            } else if (c >= a.fhi) {
                off -= uint32_t(z) * (SZ - a.fSZ[1]) + uint32_t(a.fhi) * sfa;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(st_rh, SC_LDS(st_dst + it * 4096), 16,
                                                         ok ? off : 0xFFFFFFC0u, 0, 0, 0);
            } else {
                __builtin_amdgcn_raw_ptr_buffer_load_lds(st_r, SC_LDS(st_dst + it * 4096), 16,
                                                         ok ? off : 0xFFFFFFC0u, 0, 0, 0);
            }
        } else {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(st_r, SC_LDS(st_dst + it * 4096), 16, ok ? off : a.batch_bytes,
                                                     0, 0, 0);
        }
    };
    // load it of a unit goes out in MFMA step step_of(it) of the tile before (the
    // last in the last step), behind that step's first MFMA
    constexpr int S_STEPS = R * KD * C::NKC;
    // at most one staging load per MFMA step; two where the stage is single
    // buffered ahead (NBUF = 2: each tile starts by waiting for every load and
    // store, so the order of a tile's loads does not matter)
    static_assert(S_STEPS >= C::NIT || (NBUF == 2 && 2 * S_STEPS >= C::NIT), "staging loads per MFMA step");
    // (the last load in the last step either way)
    auto step_of = [](int it) {
        return C::NIT <= S_STEPS ? ((it + 1) * S_STEPS) / C::NIT - 1 : (it * S_STEPS) / C::NIT;
    };
    // Where a group count leaves the tile's last step without epilogue stores
    // (six or more groups), a step's load goes out behind its first MFMA; else
    // after the step's epilogue piece, so that a tile's last staging load
    // follows its stores (the vmcnt waits count the stores issued after it).

    // epilogue LDS addresses: lane (g, co) writes voxel 16g + e of channel co at
    // slot (16g + e) ^ g; the read-back gives lane U = it * 64 + lane the 16 bytes
    // (voxel U / 4, channels 8 * (U % 4) ...)
    const uint32_t epi = lds0 + uint32_t(NBUF * C::STAGE_BYTES + wave * C::EPI_BYTES);
    const int co = lane & 31;
    const uint32_t ew_even = epi + uint32_t(co * 2 + 1024 * g + 64 * g);
    const uint32_t ew_odd = epi + uint32_t(co * 2 + 1024 * g - 64 * g);
    uint32_t er[2];
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int U = it * 64 + lane, v = U >> 2, uu = U & 3;
        er[it] = epi + uint32_t((v ^ ((v >> 4) & 1)) * 64 + uu * 16);
    }

    // output position of a computed tile: W tile j, output rows (o0, o1b + r)
    struct TileOut {
        int32_t j, o0, o1b, oe0;
        uint32_t nn;
        bool store;
    };
    auto tile_out = [&](const Pos& p) {
        return TileOut{p.j, org0_of(p.bz) + wz, a.org[1] + p.by * C::BY + wy * R, end0_of(p.bz), p.nn,
                       p.j >= p.jstore};
    };

    f32x16_r acc[R][KW];
    float carry[R][3];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        carry[r][0] = carry[r][1] = carry[r][2] = 0.f;
#pragma unroll
        for (int kw = 0; kw < KW; ++kw)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[r][kw][e] = 0.f;
    }

    // The epilogue of output row rr of tile t, in five pieces that the main loop
    // interleaves with the MFMAs of the next row:
    //   0, 1: out[16g + e] = A2[e] + A1[e - 1] + A0[e - 2] for e < 8, e >= 8
    //   2, 3: bf16 conversion and transpose writes to the wave's LDS buffer; 3 also
    //         issues the two read-backs
    //   4:    16-byte stores (the read-backs must have completed)
    float eo[16];
    lds_u32x4 ed[2];
    auto epi_piece = [&](int rr, int k, const TileOut& t) {
        if (k == 0) {
            // values of voxels 14, 15 of the other lane half (v_permlane32_swap with
            // itself gives lane l the row-0 value in [0] and the row-1 value in [1])
            const uint32_t x1 = __float_as_uint(acc[rr][1][15]);
            const uint32_t x2 = __float_as_uint(acc[rr][0][14]);
            const uint32_t x3 = __float_as_uint(acc[rr][0][15]);
            const auto p1 = __builtin_amdgcn_permlane32_swap(x1, x1, false, false);
            const auto p2 = __builtin_amdgcn_permlane32_swap(x2, x2, false, false);
            const auto p3 = __builtin_amdgcn_permlane32_swap(x3, x3, false, false);
            const float s1 = __uint_as_float(g ? p1[0] : p1[1]);
            const float t0 = __uint_as_float(g ? p2[0] : p2[1]);
            const float v0 = __uint_as_float(g ? p3[0] : p3[1]);
            // no voxels precede a row's first tile
            const bool row0 = t.j == 0;
            const float c1 = g ? s1 : (row0 ? 0.f : carry[rr][0]);
            const float c2 = g ? t0 : (row0 ? 0.f : carry[rr][1]);
            const float c3 = g ? v0 : (row0 ? 0.f : carry[rr][2]);
            carry[rr][0] = s1;
            carry[rr][1] = t0;
            carry[rr][2] = v0;
            if (t.j == a.NXT - 1) {
                // the row's last tile: outputs 32j + pad + 30 and + 31 would be
                // completed by a next tile whose voxels lie past the row end (zero),
                // so they are the carry terms alone (lane half 0: s1 + t0 and v0)
                const int o1 = t.o1b + rr;
                const int ox = t.j * 32 + a.pad[2] + 30;
                if (g == 0 && t.store && t.o0 < t.oe0 && o1 < a.oend[1]) {
                    __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
                        a.y + int64_t(t.nn) * a.ybatch_bytes, short(0), int(a.ybatch_bytes), 0x00020000);
                    const uint32_t rbase = uint32_t((int64_t(t.o0) * a.O[1] + o1) * a.O[2]);
                    const uint32_t cof = uint32_t(wc * 32 + co);
                    if (ox >= 0 && ox < a.O[2])
                        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, __bf16(s1 + t0)), yr,
                                                              ((rbase + uint32_t(ox)) * uint32_t(a.cout) + cof) * 2u,
                                                              0, 0);
                    if (ox + 1 >= 0 && ox + 1 < a.O[2])
                        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, __bf16(v0)), yr,
                                                              ((rbase + uint32_t(ox + 1)) * uint32_t(a.cout) + cof) * 2u,
                                                              0, 0);
                }
            }
            eo[0] = acc[rr][2][0] + c1 + c2;
            eo[1] = acc[rr][2][1] + acc[rr][1][0] + c3;
#pragma unroll
            for (int e = 2; e < 8; ++e) eo[e] = acc[rr][2][e] + acc[rr][1][e - 1] + acc[rr][0][e - 2];
        } else if (k == 1) {
#pragma unroll
            for (int e = 8; e < 16; ++e) eo[e] = acc[rr][2][e] + acc[rr][1][e - 1] + acc[rr][0][e - 2];
        } else if (k == 2 || k == 3) {
#pragma unroll
            for (int e = 8 * (k - 2); e < 8 * (k - 1); e += 2) {
                const bf16x2_r pk = {__bf16(eo[e]), __bf16(eo[e + 1])};
                const uint32_t w = __builtin_bit_cast(uint32_t, pk);
                lds_write_b16(ew_even + uint32_t(e * 64), w);
                lds_write_b16_hi(ew_odd + uint32_t((e + 1) * 64), w);
            }
            if (k == 3) {
                ed[0] = lds_read_b128(er[0]);
                ed[1] = lds_read_b128(er[1]);
            }
        } else {
            lds_ready(ed[0]);
            lds_ready(ed[1]);
            __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
                a.y + int64_t(t.nn) * a.ybatch_bytes, short(0), int(a.ybatch_bytes), 0x00020000);
            const int o1 = t.o1b + rr;
            const bool rowok = t.store && t.o0 < t.oe0 && o1 < a.oend[1];
            const uint32_t rbase = uint32_t((int64_t(t.o0) * a.O[1] + o1) * a.O[2]);
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int v = (it * 64 + lane) >> 2, uu = lane & 3;
                const int ox = t.j * 32 + a.pad[2] - (KW - 1) + v;
                const bool ok = rowok && ox >= 0 && ox < a.O[2];
                const uint32_t off =
                    ok ? ((rbase + uint32_t(ox)) * uint32_t(a.cout) + uint32_t(wc * 32 + uu * 8)) * 2u
                       : a.ybatch_bytes;
                // nontemporal (cache policy NT): the outputs are not read again
                // by this kernel (1-1.5 % faster on C3 than cached stores)
                __builtin_amdgcn_raw_buffer_store_b128(ed[it], yr, off, 0, 2);
            }
        }
    };
    // which epilogue pieces run in group q of a row
    constexpr int NG = KD * C::NKC;  // (kd, kc) groups per output row
    constexpr bool kEarlyLoad = NG >= 6;
    static_assert(NG >= 4, "five epilogue pieces in at least four groups");
    auto pieces_of = [&](int q, int rr, const TileOut& t) {
        if (NG >= 5) {
            // with six or more groups piece 4 (the stores) goes out in the MFMA
            // sequence of group 4 (see the main loop)
            if (q < (kEarlyLoad ? 4 : 5)) epi_piece(rr, q, t);
        } else {
            if (q == 0) epi_piece(rr, 0, t);
            if (q == 1) epi_piece(rr, 1, t);
            if (q == 2) {
                epi_piece(rr, 2, t);
                epi_piece(rr, 3, t);
            }
            if (q == 3) epi_piece(rr, 4, t);
        }
    };

    Pos cp{L, 0, 0, 0, 0, 0, 0}, sp{L, 0, 0, 0, 0, 0, 0};
    seg_start(cp);
    seg_start(sp);
#pragma unroll
    for (int p = 0; p < NBUF - 1; ++p) {
        stage_setup(sp, p);
#pragma unroll
        for (int it = 0; it < C::NIT; ++it) stage_load(it);
        advance(sp);
    }

    // the row R - 1 of the previous tile is pending at the start of each tile; the
    // first tile's predecessor stores nothing
    TileOut prev{0, 0, 0, 0, 0, false};
    int cbuf = 0, sbuf = NBUF - 1;
    for (uint32_t u = 0; cp.brick < a.nbricks; ++u) {
        // Unit u's loads have landed and every wave is done with the buffer that
        // is refilled next. Issued after unit u's last load: the loads of the next
        // NBUF - 2 units and the stores of the last min(u, NBUF - 2) tiles (a tile
        // body issues its staging loads last).
        const uint32_t ks = u < NBUF - 2 ? u : NBUF - 2;
        if (ks == 0)
            wait_vm_barrier<C::VM_BASE>();
        else if (ks == 1)
            wait_vm_barrier<C::VM_BASE + C::EPI_STORES>();
        else
            wait_vm_barrier<C::VM_BASE + 2 * C::EPI_STORES>();
        // the weight fragments stay in AGPRs (MFMA reads its B operand from them)
#pragma unroll
        for (int kd = 0; kd < KD; ++kd)
#pragma unroll
            for (int kh = 0; kh < KH; ++kh)
#pragma unroll
                for (int kw = 0; kw < KW; ++kw)
#pragma unroll
                    for (int kc = 0; kc < C::NKC; ++kc) asm volatile("" : "+a"(wv[kd][kh][kw][kc]));
        stage_setup(sp, sbuf);
        advance(sp);
        sbuf = sbuf + 1 == NBUF ? 0 : sbuf + 1;
        const TileOut cur = tile_out(cp);

        // steps s = (row r, group q): the KH input rows of step s + 1 are read while
        // step s multiplies
        const uint32_t boff = uint32_t(cbuf * C::STAGE_BYTES);
        constexpr int S = R * NG;
        // Step s = (row r, group q = (kd, kc)) multiplies input rows r .. r + KH - 1
        // of plane kd. Rows r + 1 .. r + KH - 1 are also the first KH - 1 rows of
        // row r + 1's step in the same group, so they stay in registers (cache[q])
        // and that step reads only its last row: R * KH reads per group become
        // KH + R - 1. Reads of step s + 1 go out while step s multiplies.
        lds_u32x4 fresh[2][KH];
        lds_u32x4 cache[NG][KH - 1];
        auto reads_of = [](int st) { return st / NG == 0 ? KH : 1; };
        auto load_step = [&](int st, lds_u32x4 (&F)[KH]) {
            const int r = st / NG, q = st % NG;
            const int kd = q / C::NKC, kc = q % C::NKC;
            if (r == 0) {
#pragma unroll
                for (int kh = 0; kh < KH; ++kh)
                    F[kh] = lds_read_b128(abase[kc] + boff + uint32_t((kd * C::IRY + kh) * C::ROW_BYTES));
            } else {
                F[0] = lds_read_b128(abase[kc] + boff + uint32_t((kd * C::IRY + r + KH - 1) * C::ROW_BYTES));
            }
        };
        load_step(0, fresh[0]);
#pragma unroll
        for (int st = 0; st < S; ++st) {
            const int cur_b = st & 1;
            const int r = st / NG, q = st % NG;
            const int kd = q / C::NKC, kc = q % C::NKC;
            if (st + 1 < S) {
                load_step(st + 1, fresh[cur_b ^ 1]);
                if (reads_of(st + 1) == KH)
                    lds_wait<KH>();
                else
                    lds_wait<1>();
            } else {
                lds_wait<0>();
            }
            lds_u32x4 A[KH];
#pragma unroll
            for (int kh = 0; kh < KH; ++kh) {
                if (r == 0) {
                    lds_ready(fresh[cur_b][kh]);
                    A[kh] = fresh[cur_b][kh];
                } else if (kh == KH - 1) {
                    lds_ready(fresh[cur_b][0]);
                    A[kh] = fresh[cur_b][0];
                } else {
                    A[kh] = cache[q][kh];
                }
            }
#pragma unroll
            for (int kh = 0; kh < KH; ++kh)
#pragma unroll
                for (int kw = 0; kw < KW; ++kw) {
                    const f32x16_r c0 = (q == 0 && kh == 0) ? f32x16_r{} : acc[r][kw];
                    acc[r][kw] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8_r, A[kh]), __builtin_bit_cast(bf16x8_r, wv[kd][kh][kw][kc]), c0,
                        0, 0, 0);
                    // the step's staging load, and in group 4 the pending row's
                    // stores, go out right behind its first MFMA, so that their issue
                    // stalls overlap that MFMA
                    if (kEarlyLoad && kh == 0 && kw == 0) {
#pragma unroll
                        for (int it = 0; it < C::NIT; ++it)
                            if (step_of(it) == st) stage_load(it);
                        if (q == 4) {
                            if (r == 0)
                                epi_piece(R - 1, 4, prev);
                            else
                                epi_piece(r - 1, 4, cur);
                        }
                    }
                }
            if constexpr (kEarlyLoad) {
                // keep that order through scheduling: one MFMA, the load, the stores,
                // the rest
                bool has_load = false;
#pragma unroll
                for (int it = 0; it < C::NIT; ++it) has_load = has_load || step_of(it) == st;
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                if (has_load) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
                if (q == 4) __builtin_amdgcn_sched_group_barrier(0x040, 2, 0);    // VMEM write
                __builtin_amdgcn_sched_group_barrier(0x008, KH * KW - 1, 0);
            }
            if (r + 1 < R) {
#pragma unroll
                for (int kh = 0; kh + 1 < KH; ++kh) cache[q][kh] = A[kh + 1];
            }
            // the pending row: R - 1 of the previous tile while row 0 multiplies,
            // else row r - 1 of this tile
            if (r == 0)
                pieces_of(q, R - 1, prev);
            else
                pieces_of(q, r - 1, cur);
            if constexpr (!kEarlyLoad) {
#pragma unroll
                for (int it = 0; it < C::NIT; ++it)
                    if (step_of(it) == st) stage_load(it);
            }
        }
        cbuf = cbuf + 1 == NBUF ? 0 : cbuf + 1;
        prev = cur;
        advance(cp);
    }
    // the last tile's row R - 1
#pragma unroll
    for (int k = 0; k < 4; ++k) epi_piece(R - 1, k, prev);
    lds_wait<0>();
    epi_piece(R - 1, 4, prev);
    // no direct loads may still target LDS when the workgroup retires
    wait_vm_barrier<0>();
}

// A folded halo the staging loads can take: margins on one axis, 0 or 1, whose
// rows are uniform over a load instruction (rpi staged rows per instruction
// share their D row, so axis 1 needs rpi == 1), 16-byte aligned slabs of < 4 GiB
// per batch item.
bool fold_fits(const Tile3& t, const Fold& f, int rpi)
{
    if (f.mask != 1u && f.mask != 2u) return false;
    const int k = f.mask == 1u ? 0 : 1;
    if (k == 1 && rpi != 1) return false;
    const int64_t SY = t.P[2] * t.c * 2;
    for (int sd = 0; sd < 2; ++sd) {
        const int64_t w = sd == 0 ? t.lo[k] : t.hi[k];
        if (reinterpret_cast<uintptr_t>(f.slab[k][sd]) % 16 != 0) return false;
        const int64_t bb = (k == 0 ? w * t.P[1] : t.P[0] * w) * SY;
        if (bb >= (int64_t(1) << 32) - 64) return false;
    }
    return true;
}

template <int CIN, int KD, int KH, int WZ, int WY, int WC, int R, int NBUF>
hipError_t launch_xm(const Tile3& t, const Conv3& cv, const void* tile, const void* wfrag, void* y, const Region& rg,
                     const Region* rg2, const Fold* fold, hipStream_t s)
{
    using C = XmCfg<CIN, KD, KH, WZ, WY, WC, R, NBUF>;
    static_assert(C::LDS_BYTES <= 160 * 1024, "LDS budget");
    XmArgs a{};
    a.fa = -1;
    if (fold) {
        if (!fold_fits(t, *fold, C::RPI)) return hipErrorNotSupported;
        a.fa = fold->mask == 1u ? 0 : 1;
        const int k = a.fa;
        a.flo = int32_t(t.lo[k]);
        a.fhi = int32_t(t.lo[k] + t.ext[k]);
        const int64_t SY = t.P[2] * t.c * 2;
        for (int sd = 0; sd < 2; ++sd) {
            const int64_t w = sd == 0 ? t.lo[k] : t.hi[k];
            // slab [P0 or w][w or P1][P2][c]: no margins on the other axes
            const int64_t sz = k == 0 ? t.P[1] * SY : w * SY;
            a.fslab[sd] = w > 0 ? fold->slab[k][sd] : nullptr;
            a.fbatch[sd] = uint32_t((k == 0 ? w : t.P[0]) * sz);
            a.fSZ[sd] = uint32_t(sz);
        }
    }
    a.tile = static_cast<const char*>(tile);
    a.wfrag = static_cast<const char*>(wfrag);
    a.y = static_cast<char*>(y);
    for (int k = 0; k < 3; ++k) {
        a.P[k] = int32_t(t.P[k]);
        a.O[k] = int32_t(cv.O[k]);
        a.pad[k] = int32_t(cv.pad[k]);
    }
    if (t.n == 0 || rg.ext[0] == 0 || rg.ext[1] == 0 || rg.ext[2] == 0) return hipSuccess;
    for (int k = 0; k < 2; ++k) {
        a.org[k] = int32_t(rg.org[k]);
        a.oend[k] = int32_t(rg.org[k] + rg.ext[k]);
    }
    a.NBZ = int32_t(ceil_div(rg.ext[0], C::BZ));
    a.nbz_a = a.NBZ;
    a.org0b = a.oend0b = 0;
    if (rg2 && rg2->ext[0] > 0) {
        a.org0b = int32_t(rg2->org[0]);
        a.oend0b = int32_t(rg2->org[0] + rg2->ext[0]);
        a.NBZ += int32_t(ceil_div(rg2->ext[0], C::BZ));
    }
    a.NBY = int32_t(ceil_div(rg.ext[1], C::BY));
    pick_raster(a.NBZ, a.NBY, 4, a.TZ, a.TY);
    a.NXT = int32_t(ceil_div(t.P[2], 32));
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t rows = t.n * int64_t(a.NBZ) * a.NBY;
    // split W rows into segments when the bricks do not fill the chip evenly
    int64_t nseg, T;
    pick_segments(rows, a.NXT, cus, 1, 4, nseg, T);
    a.nseg = int32_t(nseg);
    a.T = int32_t(T);
    const int64_t nb = rows * nseg;
    if (nb >= (int64_t(1) << 31)) return hipErrorNotSupported;
    a.nbricks = uint32_t(nb);
    a.batch_bytes = uint32_t(t.P[0] * t.P[1] * t.P[2] * t.c * 2);
    a.ybatch_bytes = uint32_t(cv.O[0] * cv.O[1] * cv.O[2] * cv.cout * 2);
    a.cout = int32_t(cv.cout);
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(nb, cus));
    auto fn = fold ? &conv_fwd_xm<CIN, KD, KH, WZ, WY, WC, R, NBUF, true>
                   : &conv_fwd_xm<CIN, KD, KH, WZ, WY, WC, R, NBUF, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       C::LDS_BYTES);
    if (e != hipSuccess) return e;
    void* args[] = {&a};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)), dim3(256), args, C::LDS_BYTES, s);
}

}  // namespace

// The W-march kernel applies to bf16, unit stride, kernel width 3 along W,
// tiles and outputs of < 4 GiB per batch item, 16-byte aligned buffers, extents
// below 2^24, the (channel, kernel) shapes instantiated below with the weight
// fragments laid out by wfrag_kernel with exactly CIN/16 chunks and cout/32
// tiles, and a folded halo that fold_fits.
bool conv_fwd_rows_supported(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                             const void* wfrag, int nkc_frag, int nt_frag, const void* y, const Fold* fold)
{
    if (dt != SHARD_BF16 || force_tiled()) return false;
    if (cv.S[0] != 1 || cv.S[1] != 1 || cv.S[2] != 1 || cv.K[2] != 3) return false;
    if (reinterpret_cast<uintptr_t>(tile) % 16 != 0 || reinterpret_cast<uintptr_t>(wfrag) % 16 != 0 ||
        reinterpret_cast<uintptr_t>(y) % 16 != 0)
        return false;
    const int64_t bb = t.P[0] * t.P[1] * t.P[2] * t.c * 2;
    const int64_t yb = cv.O[0] * cv.O[1] * cv.O[2] * cv.cout * 2;
    if (bb >= (int64_t(1) << 32) - 64 || yb >= (int64_t(1) << 32) - 64) return false;
    for (int k = 0; k < 3; ++k)
        if (std::abs(cv.pad[k]) > (1 << 20) || cv.O[k] >= (int64_t(1) << 24) || t.P[k] >= (int64_t(1) << 24))
            return false;
    int rpi = 0;
    if (t.c == 32 && cv.cout == 32 && cv.K[0] == 3 && cv.K[1] == 3 && nkc_frag == 2 && nt_frag == 1) rpi = 2;
    if (t.c == 64 && cv.cout == 64 && cv.K[0] == 1 && cv.K[1] == 3 && nkc_frag == 4 && nt_frag == 2) rpi = 1;
    if (rpi == 0) return false;
    return !fold || fold_fits(t, *fold, rpi);
}

// Launches a region of a call conv_fwd_rows_supported accepts (regions cut axes
// 0 and 1 only: the W march covers whole rows); hipErrorNotSupported otherwise.
hipError_t launch_conv_fwd_rows(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                const void* wfrag, int nkc_frag, int nt_frag, void* y, const Region& rg,
                                const Fold* fold, hipStream_t s, const Region* rg2)
{
    if (!conv_fwd_rows_supported(t, cv, dt, tile, wfrag, nkc_frag, nt_frag, y, fold)) return hipErrorNotSupported;
    if (rg.org[2] != 0 || rg.ext[2] != cv.O[2]) return hipErrorNotSupported;
    if (rg2) {
        // a second region must differ from the first along axis 0 only, and not overlap it
        if (rg2->org[1] != rg.org[1] || rg2->ext[1] != rg.ext[1] || rg2->org[2] != rg.org[2] ||
            rg2->ext[2] != rg.ext[2] || (rg2->org[0] < rg.org[0] + rg.ext[0] && rg.org[0] < rg2->org[0] + rg2->ext[0]))
            return hipErrorNotSupported;
    }
    const int64_t ext0 = std::max<int64_t>(rg.ext[0], rg2 ? rg2->ext[0] : 0);
    if (t.c == 32) {
        // thin regions along axis 0 (the boundary planes of a D-sharded tile) take
        // bricks one plane deep (8 rows high; the stage of 30 input rows fits LDS
        // twice) or two; per-output arithmetic is the same in all
        if (ext0 == 1) return launch_xm<32, 3, 3, 1, 4, 1, 2, 2>(t, cv, tile, wfrag, y, rg, rg2, fold, s);
        if (ext0 <= 2) return launch_xm<32, 3, 3, 2, 2, 1, 2, 3>(t, cv, tile, wfrag, y, rg, rg2, fold, s);
        return launch_xm<32, 3, 3, 4, 1, 1, 2, 3>(t, cv, tile, wfrag, y, rg, rg2, fold, s);
    }
    // thin regions along axis 1 (the boundary rows of an H-sharded 2D tile)
    if (rg.ext[1] <= 2) return launch_xm<64, 1, 3, 1, 2, 2, 2, 3>(t, cv, tile, wfrag, y, rg, rg2, fold, s);
    return launch_xm<64, 1, 3, 1, 2, 2, 4, 3>(t, cv, tile, wfrag, y, rg, rg2, fold, s);
}

}  // namespace shardconv
