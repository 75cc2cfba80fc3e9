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
// tile[box] += slab (dense), element-wise in binary32; esz 2 (bf16) or 4 (f32).
hipError_t launch_box_add(const BoxCopy& b, int esz, const void* slab, void* tile, hipStream_t s);

// Where a forward convolution writes output (n, o0, o1, o2, co): element
// base + n*str[0] + o0*str[1] + o1*str[2] + o2*str[3] + co. The dense map of
// Conv3 is y[n][O0][O1][O2][cout]; the input gradient of a strided convolution
// writes each stride phase into every S-th row of the tile with a strided map.
struct OutMap {
    int64_t base;
    int64_t str[4];
};
OutMap dense_out(const Conv3& cv);

// Convolution launchers. `ws` holds at least conv_*_workspace(...) bytes.
size_t conv_fwd_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
size_t conv_wgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_conv_fwd(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* w,
                           void* y, void* ws, hipStream_t s);
// The same with an output map (a non-dense map takes the general kernels).
hipError_t launch_conv_fwd_mapped(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                  const void* w, void* y, const OutMap& om, void* ws, hipStream_t s);
hipError_t launch_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                             float* dw, void* ws, hipStream_t s);
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
hipError_t launch_conv_fwd_rows(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                const void* wfrag, int nkc_frag, int nt_frag, void* y, hipStream_t s);
size_t wgrad_xm_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_wgrad_xm(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* dw, void* ws, hipStream_t s);
size_t wgrad_tr_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt);
hipError_t launch_wgrad_tr(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                           float* part, int32_t red[6], hipStream_t s);

// Which implementation a call takes, read from the environment variable
// SHARDCONV_ALGO at each call: unset picks the fastest applicable kernel,
// "tiled" skips the shape-specialised kernels, "generic" forces the plain
// direct kernels (tests use both to cross-check the kernels against each other).
bool force_generic();
bool force_tiled();

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

}  // namespace shardconv
