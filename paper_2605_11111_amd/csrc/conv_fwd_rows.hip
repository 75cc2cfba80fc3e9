// Forward convolution, bf16, for unit stride and small weight sets (the
// halo-padded 3D/2D shard workloads): a persistent implicit GEMM whose operands
// never leave the CU between reuses.
//
//  * One workgroup per CU (4 waves) sweeps output bricks of WZ x (WY*R) x 32
//    voxels. The whole weight set, pre-arranged in MFMA B-fragment order, sits
//    in LDS for the workgroup's lifetime.
//  * The input footprint of a brick (the brick grown by the kernel reach; the
//    halo rows arrive this way) is staged in 16-channel chunks by direct
//    global->LDS buffer loads (no VGPR round trip), double buffered: the next
//    chunk streams in while the current one feeds the MFMAs. Voxels outside the
//    tile load as zero (out-of-range buffer offsets), which is the zero padding.
//  * Each wave owns R consecutive output rows of one plane (32 voxels each, an
//    M tile of v_mfma_f32_32x32x16_bf16). For a fixed (kd, kw) the A fragment of
//    input row j serves output rows j - kh for every kh, so R + KH - 1 LDS reads
//    feed R * KH MFMAs.
//  * LDS addresses are per-lane constants plus compile-time immediates; the
//    16-byte unit of a voxel is XOR-swizzled by bit 3 of its x position so the
//    16 lanes of a ds_read_b128 phase hit 16 distinct bank groups.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_r;
typedef __attribute__((ext_vector_type(16))) float f32x16_r;

#define SC_LDS(p) ((__attribute__((address_space(3))) void*)(p))

namespace {

struct RowsArgs {
    const char* tile;
    const char* wfrag;
    char* y;
    int64_t n;
    int64_t P[3], O[3];
    int32_t pad[3];
    int32_t NB[3];
    int64_t nbricks;
    uint32_t batch_bytes;   // tile bytes per batch item (< 2^32)
    int32_t cout;
};

template <int CIN, int NT, int KD, int KH, int KW, int WZ, int WY, int R>
struct RowsCfg {
    static constexpr int NKC = CIN / 16;          // 16-channel K chunks
    static constexpr int BZ = WZ, BY = WY * R, BX = 32;
    static constexpr int BIZ = BZ + KD - 1, BIY = BY + KH - 1, BIX = BX + KW - 1;
    static constexpr int BIV = BIZ * BIY * BIX;
    static constexpr int SLOTS = BIV * 2;          // 16-byte units per chunk
    static constexpr int SLOTS_PAD = (SLOTS + 255) / 256 * 256;
    static constexpr int NIT = SLOTS_PAD / 256;    // direct-load instructions per thread per chunk
    static constexpr int CHUNK_BYTES = SLOTS_PAD * 16;
    static constexpr int TAPS = KD * KH * KW;
    static constexpr int W_BYTES = TAPS * NKC * NT * 1024;
    static constexpr int W_SLOTS = W_BYTES / 16;
    static constexpr int LDS_BYTES = W_BYTES + 2 * CHUNK_BYTES;
    static constexpr int NROWS_IN = R + KH - 1;    // input rows a wave reads per (kd, kw)
};

template <int CIN, int NT, int KD, int KH, int KW, int WZ, int WY, int R>
__global__ __launch_bounds__(256, 1) void conv_fwd_rows(RowsArgs a)
{
    using C = RowsCfg<CIN, NT, KD, KH, KW, WZ, WY, R>;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    char* wl = lds;                       // weights
    char* cb0 = lds + C::W_BYTES;         // chunk buffer 0 (buffer 1 follows)
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wz = wave / WY, wy = wave % WY;
    const int g = lane >> 5;
    const int ox = lane & 31;
    const int64_t nblk_grid = gridDim.x;
    const int64_t L = xcd_remap(blockIdx.x, nblk_grid);

    // weights -> LDS (once)
    {
        __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.wfrag), short(0),
                                                                      C::W_BYTES, 0x00020000);
        for (int s0 = 0; s0 < C::W_SLOTS; s0 += 256) {
            const int s = s0 + tid;
            if (s < C::W_SLOTS)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, SC_LDS(wl + (s0 + wave * 64) * 16), 16, s * 16, 0, 0, 0);
        }
    }

    // per-thread staging slots: relative byte offset within a brick and its (z, y, x)
    uint32_t srel[C::NIT];
    uint32_t szyx[C::NIT];  // z << 20 | y << 10 | x, or 0xffffffff for padding slots
#pragma unroll
    for (int it = 0; it < C::NIT; ++it) {
        const int s = it * 256 + tid;
        if (s < C::SLOTS) {
            const int v = s >> 1;
            const int x = v % C::BIX;
            const int yz = v / C::BIX;
            const int y = yz % C::BIY;
            const int z = yz / C::BIY;
            const int u = (s & 1) ^ ((x >> 3) & 1);
            srel[it] = uint32_t(((int64_t(z) * a.P[1] + y) * a.P[2] + x) * (CIN * 2) + u * 16);
            szyx[it] = (uint32_t(z) << 20) | (uint32_t(y) << 10) | uint32_t(x);
        } else {
            srel[it] = 0;
            szyx[it] = 0xffffffffu;
        }
    }

    // per-lane A-read base (byte address within chunk buffer 0) for each kw
    uint32_t abase[KW];
#pragma unroll
    for (int kw = 0; kw < KW; ++kw) {
        const int x = ox + kw;
        abase[kw] = uint32_t((wz * C::BIY + wy * R) * C::BIX * 32 + x * 32 + ((g ^ ((x >> 3) & 1)) * 16)) +
                    uint32_t(C::W_BYTES);
    }
    const uint32_t bbase = uint32_t(lane * 16);

    const int64_t per_b = (a.nbricks - L + nblk_grid - 1) / nblk_grid;  // bricks of this workgroup
    const int64_t nchunks = per_b * C::NKC;

    // stage chunk q (brick index it_b = q / NKC, channel chunk kc = q % NKC) into buffer q & 1
    auto stage = [&](int64_t q) {
        const int64_t bi = L + (q / C::NKC) * nblk_grid;
        const int kc = int(q % C::NKC);
        int64_t b = bi;
        const int bx = int(b % a.NB[2]);
        b /= a.NB[2];
        const int by = int(b % a.NB[1]);
        b /= a.NB[1];
        const int bz = int(b % a.NB[0]);
        const int64_t nn = b / a.NB[0];
        const int64_t i0 = int64_t(bz) * C::BZ - a.pad[0];
        const int64_t i1 = int64_t(by) * C::BY - a.pad[1];
        const int64_t i2 = int64_t(bx) * C::BX - a.pad[2];
        const bool inner = i0 >= 0 && i0 + C::BIZ <= a.P[0] && i1 >= 0 && i1 + C::BIY <= a.P[1] && i2 >= 0 &&
                           i2 + C::BIX <= a.P[2];
        __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(a.tile) + nn * int64_t(a.batch_bytes), short(0), int(a.batch_bytes), 0x00020000);
        const int64_t origin = ((i0 * a.P[1] + i1) * a.P[2] + i2) * (CIN * 2) + kc * 32;
        char* dst = cb0 + (q & 1) * C::CHUNK_BYTES;
#pragma unroll
        for (int it = 0; it < C::NIT; ++it) {
            const uint32_t zyx = szyx[it];
            if (zyx == 0xffffffffu) continue;
            uint32_t off;
            if (inner) {
                off = uint32_t(origin + srel[it]);
            } else {
                const int64_t t0 = i0 + (zyx >> 20), t1 = i1 + ((zyx >> 10) & 1023), t2 = i2 + (zyx & 1023);
                const bool ok = t0 >= 0 && t0 < a.P[0] && t1 >= 0 && t1 < a.P[1] && t2 >= 0 && t2 < a.P[2];
                off = ok ? uint32_t(origin + int64_t(srel[it])) : a.batch_bytes;
            }
            __builtin_amdgcn_raw_ptr_buffer_load_lds(r, SC_LDS(dst + (it * 256 + wave * 64) * 16), 16, off, 0, 0, 0);
        }
    };

    f32x16_r acc[R][NT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[r][t][e] = 0.f;

    if (nchunks > 0) stage(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    bf16_t* y = reinterpret_cast<bf16_t*>(a.y);
    for (int64_t q = 0; q < nchunks; ++q) {
        if (q + 1 < nchunks) stage(q + 1);
        const int kc = int(q % C::NKC);
        const uint32_t boff = uint32_t((q & 1) * C::CHUNK_BYTES);
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) {
#pragma unroll
            for (int kw = 0; kw < KW; ++kw) {
                uint4 av[C::NROWS_IN];
#pragma unroll
                for (int j = 0; j < C::NROWS_IN; ++j)
                    av[j] = *reinterpret_cast<const uint4*>(lds + abase[kw] + boff +
                                                            (kd * C::BIY + j) * C::BIX * 32);
                uint4 bv[KH][NT];
#pragma unroll
                for (int kh = 0; kh < KH; ++kh)
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const int tap = (kd * KH + kh) * KW + kw;
                        bv[kh][t] = *reinterpret_cast<const uint4*>(wl + bbase + ((tap * C::NKC + kc) * NT + t) * 1024);
                    }
#pragma unroll
                for (int kh = 0; kh < KH; ++kh)
#pragma unroll
                    for (int r = 0; r < R; ++r)
#pragma unroll
                        for (int t = 0; t < NT; ++t)
                            acc[r][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                __builtin_bit_cast(bf16x8_r, av[r + kh]), __builtin_bit_cast(bf16x8_r, bv[kh][t]),
                                acc[r][t], 0, 0, 0);
            }
        }
        if (kc == C::NKC - 1) {
            // epilogue of brick q / NKC: rows 8*(e/4) + 4*g + (e%4) of each M tile, column = output channel
            const int64_t bi = L + (q / C::NKC) * nblk_grid;
            int64_t b = bi;
            const int bx = int(b % a.NB[2]);
            b /= a.NB[2];
            const int by = int(b % a.NB[1]);
            b /= a.NB[1];
            const int bz = int(b % a.NB[0]);
            const int64_t nn = b / a.NB[0];
            const int64_t o0 = int64_t(bz) * C::BZ + wz;
            const int64_t ox0 = int64_t(bx) * C::BX;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int64_t o1 = int64_t(by) * C::BY + wy * R + r;
                const bool rok = o0 < a.O[0] && o1 < a.O[1];
                bf16_t* row = y + (((nn * a.O[0] + o0) * a.O[1] + o1) * a.O[2] + ox0) * a.cout;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int co = t * 32 + ox;  // lane's column
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int xr = 8 * (e >> 2) + 4 * g + (e & 3);
                        if (rok && ox0 + xr < a.O[2] && co < a.cout)
                            row[xr * a.cout + co] = __builtin_bit_cast(bf16_t, __bf16(acc[r][t][e]));
                        acc[r][t][e] = 0.f;
                    }
                }
            }
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }
}

template <int CIN, int NT, int KD, int KH, int KW, int WZ, int WY, int R>
hipError_t launch_rows(const Tile3& t, const Conv3& cv, const void* tile, const void* wfrag, void* y, hipStream_t s)
{
    using C = RowsCfg<CIN, NT, KD, KH, KW, WZ, WY, R>;
    RowsArgs a{};
    a.tile = static_cast<const char*>(tile);
    a.wfrag = static_cast<const char*>(wfrag);
    a.y = static_cast<char*>(y);
    a.n = t.n;
    for (int k = 0; k < 3; ++k) {
        a.P[k] = t.P[k];
        a.O[k] = cv.O[k];
        a.pad[k] = int32_t(cv.pad[k]);
    }
    const int bo[3] = {C::BZ, C::BY, C::BX};
    for (int k = 0; k < 3; ++k) a.NB[k] = int32_t(ceil_div(cv.O[k], bo[k]));
    a.nbricks = t.n * int64_t(a.NB[0]) * a.NB[1] * a.NB[2];
    a.batch_bytes = uint32_t(t.P[0] * t.P[1] * t.P[2] * t.c * 2);
    a.cout = int32_t(cv.cout);
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(a.nbricks, cus));
    auto fn = &conv_fwd_rows<CIN, NT, KD, KH, KW, WZ, WY, R>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       C::LDS_BYTES);
    if (e != hipSuccess) return e;
    void* args[] = {&a};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)), dim3(256), args, C::LDS_BYTES, s);
}

}  // namespace

// The row-reuse kernel applies to bf16, unit stride, tiles of < 4 GiB per batch
// item, 16-byte aligned tiles, and the (channel, kernel) shapes instantiated below.
// Returns hipErrorNotSupported when it does not apply.
hipError_t launch_conv_fwd_rows(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                const void* wfrag, int nkc_frag, int nt_frag, void* y, hipStream_t s)
{
    if (dt != SHARD_BF16 || force_tiled()) return hipErrorNotSupported;
    if (cv.S[0] != 1 || cv.S[1] != 1 || cv.S[2] != 1) return hipErrorNotSupported;
    if (reinterpret_cast<uintptr_t>(tile) % 16 != 0 || reinterpret_cast<uintptr_t>(wfrag) % 16 != 0)
        return hipErrorNotSupported;
    const int64_t bb = t.P[0] * t.P[1] * t.P[2] * t.c * 2;
    if (bb >= (int64_t(1) << 32) - 64) return hipErrorNotSupported;
    for (int k = 0; k < 3; ++k)
        if (std::abs(cv.pad[k]) > (1 << 20) || cv.O[k] > (int64_t(1) << 30)) return hipErrorNotSupported;
    // fragment arrays laid out by wfrag_kernel with exactly CIN/16 chunks and NT tiles
    if (t.c == 32 && cv.cout == 32 && cv.K[0] == 3 && cv.K[1] == 3 && cv.K[2] == 3 && nkc_frag == 2 && nt_frag == 1)
        return launch_rows<32, 1, 3, 3, 3, 4, 1, 4>(t, cv, tile, wfrag, y, s);
    if (t.c == 64 && cv.cout == 64 && cv.K[0] == 1 && cv.K[1] == 3 && cv.K[2] == 3 && nkc_frag == 4 && nt_frag == 2)
        return launch_rows<64, 2, 1, 3, 3, 1, 4, 4>(t, cv, tile, wfrag, y, s);
    return hipErrorNotSupported;
}

}  // namespace shardconv
