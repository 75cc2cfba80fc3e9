// Internal interfaces between the C-ABI layer (api.cpp) and the HIP kernels.
// Every public call is normalised to three spatial axes: a 2D problem gets a
// leading unit axis and a 1D problem two, with kernel 1, stride 1, pad 0 there.
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime.h>

#include "shardconv.h"

namespace shardconv {

// A padded tile: dense [n][P0][P1][P2][c], all sizes in elements.
struct Tile3 {
    int64_t n, c;
    int64_t P[3];                 // padded extents
    int64_t lo[3], ext[3], hi[3]; // margins and interior
    int esz;                      // bytes per element (2 or 4)
};

// A convolution read off a padded tile (see shard_conv_fwd).
struct Conv3 {
    int64_t cout;
    int64_t K[3], S[3], pad[3], O[3];
    int64_t taps() const { return K[0] * K[1] * K[2]; }
    int64_t out_voxels() const { return O[0] * O[1] * O[2]; }
};

// A box copy between a tile and a dense slab (pack, unpack, zero fill).
// After merging contiguous inner axes the box is `rows` = c0*c1*c2 runs of
// `run` bytes; run r = (i0, i1, i2) starts at tile byte offset
// base + i0*t0 + i1*t1 + i2*t2 and at slab byte offset r*run.
struct BoxCopy {
    int64_t base;
    int64_t cnt[3];
    int64_t tstride[3];
    int64_t run;
};

enum CopyDir { TILE_TO_SLAB = 0, SLAB_TO_TILE = 1, ZERO_TILE = 2 };

hipError_t launch_box_copy(const BoxCopy& b, CopyDir dir, const void* src, void* dst, hipStream_t s);
// n (1 or 2) box copies in one launch (both faces or margins of an axis).
hipError_t launch_box_copies(const BoxCopy* const* b, const CopyDir* dir, const void* const* src, void* const* dst,
                             int n, hipStream_t s);
// tile[box] += slab (dense), element-wise in binary32; esz 2 (bf16) or 4 (f32).
hipError_t launch_box_add(const BoxCopy& b, int esz, const void* slab, void* tile, hipStream_t s);
// n (1 or 2) non-overlapping box adds in one launch (both faces of an axis).
hipError_t launch_box_adds(const BoxCopy* const* b, int esz, const void* const* slab, void* tile, int n,
                           hipStream_t s);

// Where a forward convolution writes output (n, o0, o1, o2, co): element
// base + n*str[0] + o0*str[1] + o1*str[2] + o2*str[3] + co. The dense map of
// Conv3 is y[n][O0][O1][O2][cout]; the input gradient of a strided convolution
// writes each stride phase into every S-th row of the tile with a strided map.
struct OutMap {
    int64_t base;
    int64_t str[4];
};
OutMap dense_out(const Conv3& cv);

// A convolution whose halo is folded into its tile loads: the margin rows of
// the padded tile are not read; a voxel in a margin comes from the slab received
// for that margin (laid out as shard_halo_slab_shape gives: padded extents on
// earlier axes, the margin width on its own axis, the interior on later axes) or
// is zero where no slab is given (a global boundary). Axes are resolved from the
// last to the first, so a corner voxel comes from the later axis's slab, as
// after unpacking the slabs in ascending axis order. `mask` has bit k set for
// every axis with a margin.
struct Fold {
    const char* slab[3][2];
    int64_t lo[3], ext[3], P[3];
    uint32_t mask;
};

// Byte offset of voxel (nn, t0, t1, t2) of a padded tile of `vox_bytes` bytes
// per voxel, and the buffer it lies in (the tile, a slab, or null for zero).
__host__ __device__ inline const char* fold_voxel(const Fold& f, const char* tile, int64_t nn, int64_t t0, int64_t t1,
                                                  int64_t t2, int64_t vox_bytes)
{
    const int64_t tc[3] = {t0, t1, t2};
    for (int a = 2; a >= 0; --a) {
        if (!((f.mask >> a) & 1u)) continue;
        const bool in_lo = tc[a] < f.lo[a];
        const bool in_hi = tc[a] >= f.lo[a] + f.ext[a];
        if (!in_lo && !in_hi) continue;
        const char* slab = f.slab[a][in_hi ? 1 : 0];
        if (!slab) return nullptr;
        int64_t e[3], c[3];
        for (int b = 0; b < 3; ++b) {
            if (b < a) {
                e[b] = f.P[b];
                c[b] = tc[b];
            } else if (b == a) {
                e[b] = in_hi ? f.P[a] - f.lo[a] - f.ext[a] : f.lo[a];
                c[b] = in_hi ? tc[a] - f.lo[a] - f.ext[a] : tc[a];
            } else {
                e[b] = f.ext[b];
                c[b] = tc[b] - f.lo[b];
            }
        }
        return slab + (((nn * e[0] + c[0]) * e[1] + c[1]) * e[2] + c[2]) * vox_bytes;
    }
    return tile + (((nn * f.P[0] + t0) * f.P[1] + t1) * f.P[2] + t2) * vox_bytes;
}

// The outputs a call computes: the box [org, org + ext) of the owned outputs
// (Conv3::O); the output map stays that of the whole owned box.
struct Region {
    int64_t org[3], ext[3];
};

// Convolution launchers. `ws` holds at least conv_*_workspace(...) bytes.
size_t conv_fwd_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
size_t conv_wgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_conv_fwd(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* w,
                           void* y, void* ws, hipStream_t s);
// The same with an output map (a non-dense map takes the general kernels).
hipError_t launch_conv_fwd_mapped(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                  const void* w, void* y, const OutMap& om, void* ws, hipStream_t s);
// The kernel family a forward call takes. Every region of one call takes the
// same family, so an output is summed in the same order whichever region
// computes it.
enum FwdFamily { FWD_GENERIC = 0, FWD_TILED = 1, FWD_ROWS = 2 };
FwdFamily fwd_family(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* y,
                     const OutMap& om, const Fold* fold, const void* ws);
// A region of the outputs on a chosen family, with the halo folded into the
// loads when `fold` is given. `frags_ready`: ws already holds the weight
// fragments (an earlier region of the same call with the same weights laid
// them out), so they are not laid out again.
hipError_t launch_conv_fwd_region(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                  const void* w, void* y, const OutMap& om, const Region& rg, const Fold* fold,
                                  FwdFamily fam, void* ws, hipStream_t s,
                                  bool frags_ready = false);
// Two regions that differ along axis 0 only, in one launch of the W-march
// kernel (FWD_ROWS); hipErrorNotSupported when that kernel cannot take them
// together (nothing launched).
hipError_t launch_conv_fwd_region_pair(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                       const void* w, void* y, const Region& ra, const Region& rb, const Fold* fold,
                                       void* ws, hipStream_t s, bool frags_ready);
// n (2 to 4) regions in one launch of the tiled kernel (FWD_TILED), each with
// bricks of its own shape; hipErrorNotSupported when their plans take
// different kernels (nothing launched).
hipError_t launch_conv_fwd_tiled_group(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                       const void* w, void* y, const OutMap& om, const Region* rs, int n,
                                       const Fold* fold, void* ws, hipStream_t s, bool frags_ready);
// The forward with its workspace in the library's per-device scratch array
// (noalloc.hip): bytes it holds, and the launch (the caller has checked that
// conv_fwd_workspace fits).
size_t conv_fwd_noalloc_limit();
hipError_t launch_conv_fwd_noalloc(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                   const void* w, void* y, hipStream_t s);
hipError_t launch_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                             float* dw, void* ws, hipStream_t s);
// The same with the halo folded into the loads (the kernels that cannot fold
// are passed over).
hipError_t launch_conv_wgrad_folded(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                    const void* dy, float* dw, void* ws, const Fold& fold, hipStream_t s);
size_t conv_dgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_conv_dgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* dy, const void* w,
                             void* dtile, void* ws, hipStream_t s);

// Group normalisation of a shard's interior (see norm.hip).
size_t norm_workspace(const Tile3& t, int64_t groups);
hipError_t launch_norm_stats(const Tile3& t, shard_dtype_t dt, const void* tile, int64_t groups, double* sums,
                             void* ws, hipStream_t s);
hipError_t launch_norm_apply(const Tile3& t, shard_dtype_t dt, const void* tile, const double* sums, double count,
                             double eps, int64_t groups, const float* gamma, const float* beta, void* out, void* ws,
                             hipStream_t s);

// Specialised kernels; each returns hipErrorNotSupported when the shape is
// outside what it handles (the caller then takes the general kernel).
bool conv_fwd_rows_supported(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                             const void* wfrag, int nkc_frag, int nt_frag, const void* y, const Fold* fold);
// rg2 (optional): a second region in the same launch, differing from rg along
// axis 0 only and not overlapping it; hipErrorNotSupported otherwise.
hipError_t launch_conv_fwd_rows(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                const void* wfrag, int nkc_frag, int nt_frag, void* y, const Region& rg,
                                const Fold* fold, hipStream_t s, const Region* rg2 = nullptr);
size_t wgrad_xm_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
// `status`: the call's status word (see kWgradStatusBytes).
hipError_t launch_wgrad_xm(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* dw, void* ws, const Fold* fold, uint32_t* status, hipStream_t s);
size_t wgrad_tr_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_wgrad_tr(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* part, int32_t red[6], hipStream_t s);

// Options of the calling host thread (shard_set_call_opts): which kernel family
// a convolution takes - the fastest applicable (default), the general tiled MFMA
// kernels past the shape-specialised ones, or the plain direct kernels (tests
// cross-check the families against each other) - and the poll bound of the
// weight gradient's inter-wave hand-off waits (0: the default).
struct CallOpts {
    int32_t kernels;
    uint32_t wait_polls;
};
const CallOpts& call_opts();
bool force_generic();
bool force_tiled();

// The weight-gradient workspace starts with a status block: its first 32-bit
// word is 0 after a call completed normally and nonzero when a bounded wait of
// the kernel gave up (dw then holds NaN); bytes [kWgradZeroOff, +64) are zeros,
// a source for loads of zero padding. Cleared by every call.
constexpr size_t kWgradStatusBytes = 256;
constexpr size_t kWgradZeroOff = 64;
constexpr uint32_t kDefaultWaitPolls = 1u << 20;
hipError_t launch_wgrad_status_clear(uint32_t* status, hipStream_t s);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

}  // namespace shardconv
