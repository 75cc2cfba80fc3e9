/*
 * shardconv - the per-shard hot path of domain-parallel convolution on one
 * MI355X (gfx950) GPU.
 *
 * In domain parallelism a tensor [B][C][spatial...] is split along its spatial
 * axes below batch size one (ShardTensor paper, section "Introduction"). Each
 * shard owns a box of the input with arbitrary per-rank extents (section
 * "ShardTensor", Table 2, "sharding shapes"). A convolution on a shard first
 * fetches the adjacent rows ("halo") from its neighbours so that it is
 * numerically consistent with the unsharded operation (section "PyTorch
 * Dispatch"), and because a convolution changes the global shape its output
 * chunks are uneven (section "ShardTensor"). This library implements that
 * per-shard work:
 *
 *   shard_conv_geometry   which outputs a shard owns and the halo it needs (host)
 *   shard_halo_pack       copy a boundary face of the tile into a dense slab
 *   shard_halo_unpack     copy a received slab into a margin, or zero-fill it
 *   shard_halo_pack_pair, shard_halo_unpack_pair
 *                         both faces / both margins of an axis in one launch
 *   shard_conv_fwd        convolution read off the padded tile
 *   shard_conv_wgrad      the shard's partial weight gradient
 *   shard_conv_interior   outputs that need no halo (host only)
 *   shard_conv_fwd_folded forward reading the halo from the received slabs,
 *                         all outputs or the interior / boundary part
 *   shard_conv_wgrad_folded
 *                         weight gradient reading the halo from the slabs
 *   shard_conv_dgrad      the input gradient read back onto the padded tile
 *   shard_halo_pack_margin, shard_halo_accumulate
 *                         the reverse halo exchange of the backward pass
 *   shard_halo_pack_margin_pair, shard_halo_accumulate_pair
 *                         both sides of an axis's reverse exchange in one launch
 *   shard_norm_stats, shard_norm_apply
 *                         group normalisation with statistics over all shards
 *   shard_attn_block      one block step of ring attention (log-space merge)
 *
 * Convolution semantics are PyTorch's cross-correlation (no bias, dilation 1,
 * groups 1), which the paper's programming model keeps (section "Benchmarks
 * and Applications", Algorithm 1, step 4).
 *
 * Conventions shared by every call:
 *  - Spatial axes are numbered outermost first (3D: D=0, H=1, W=2; 2D: H=0,
 *    W=1). Entries of per-axis arrays at index >= ndim are ignored.
 *  - A padded tile is dense, channels-last:
 *        [n][P0][P1][P2][c],  P_a = halo_lo[a] + ext[a] + halo_hi[a]
 *    (axes >= ndim have extent 1). Row halo_lo[a] of axis a is the shard's
 *    first interior row; the margins hold neighbour rows (or zero padding at a
 *    global boundary).
 *  - Activations (tile, y, dy, slabs) are SHARD_F32 (binary32) or SHARD_BF16
 *    (bfloat16); weights w have the activation dtype; dw is always binary32.
 *    Convolutions accumulate in binary32; a bf16 y is rounded to nearest-even
 *    from the binary32 sum.
 *  - Every device pointer is owned by the caller. The library never allocates,
 *    frees or synchronises; every device call is enqueued on `stream` and
 *    returns immediately. Buffers must not overlap.
 *  - Every argument is checked on the host before any launch; on an error
 *    nothing is written. No exception crosses this interface, and the library
 *    keeps no mutable global state: the only state is the calling host thread's
 *    own options (shard_set_call_opts), so calls from several host threads are
 *    safe.
 *  - Device pointers must be aligned to their element size (2 or 4 bytes);
 *    16-byte aligned buffers take the vectorised paths.
 */
#ifndef SHARDCONV_H
#define SHARDCONV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SHARD_OK = 0,
    SHARD_ERR_INVALID = 1,      /* a malformed argument (null pointer, negative size, bad axis, ...) */
    SHARD_ERR_UNSUPPORTED = 2,  /* well formed but outside what is implemented (see each call) */
    SHARD_ERR_HIP = 3           /* the HIP runtime rejected a launch */
} shard_status_t;

typedef enum { SHARD_F32 = 0, SHARD_BF16 = 1 } shard_dtype_t;

/* Descriptor of a padded tile (see the layout above). ndim in {1, 2, 3};
 * n >= 0 batch items, c >= 1 channels, ext[a] >= 0 interior rows,
 * halo_lo[a], halo_hi[a] >= 0 margin rows. */
typedef struct {
    int32_t ndim;
    int64_t n, c;
    int64_t ext[3];
    int64_t halo_lo[3], halo_hi[3];
} shard_tile_t;

/*
 * Geometry of one shard (host only, no device work).
 *
 * Per axis a: the full domain has global_ext[a] rows; this shard's interior is
 * [shard_off[a], shard_off[a] + shard_ext[a]); kernel[a] is odd, stride[a] >= 1;
 * the convolution pads the full domain with P = (kernel - 1) / 2 zeros per side
 * ("same" padding), so the full output has (G + 2P - K) / S + 1 rows.
 * Output j is owned by the shard whose interior contains its anchor j*S (the
 * reading this library takes of the paper's uneven output chunks).
 *
 * Outputs per axis:
 *   out_off, out_ext  the owned output rows [out_off, out_off + out_ext) of the
 *                     full output (out_ext may be 0: the shard owns nothing);
 *   halo_lo, halo_hi  margin rows the padded tile needs below / above the
 *                     interior; on a sharded axis margins outside the domain are
 *                     zero padding (unpack with slab = NULL), on an unsharded
 *                     axis (sharded_mask[a] == 0, shard_off 0, shard_ext = G)
 *                     they are 0;
 *   pad_lo            the value to pass to shard_conv_fwd/wgrad: P on unsharded
 *                     axes; on sharded axes <= 0, negative when the first owned
 *                     output's window starts inside the interior (stride > P+1).
 * Errors: SHARD_ERR_INVALID for null pointers, ndim outside 1..3,
 * non-positive kernel, stride < 1, global_ext < 1, or an interior box outside
 * the domain (or not the whole axis when unsharded); SHARD_ERR_UNSUPPORTED for
 * an even kernel (no symmetric "same" padding) when the rest is well formed.
 */
shard_status_t shard_conv_geometry(int32_t ndim, const int64_t global_ext[], const int64_t shard_off[],
                                   const int64_t shard_ext[], const int64_t kernel[], const int64_t stride[],
                                   const int64_t sharded_mask[], int64_t halo_lo[], int64_t halo_hi[],
                                   int64_t pad_lo[], int64_t out_off[], int64_t out_ext[]);

/*
 * Shape of the slab exchanged along `axis` with the given width: writes
 * shape_out[5] = {n, s0, s1, s2, c} with s_axis = width, s_b the padded extent
 * for b < axis and the interior extent for b > axis (axes are exchanged in
 * ascending order, so a slab carries the corner rows of every earlier axis),
 * and 1 for b >= ndim. The slab is dense in that order. Host only.
 * Errors: SHARD_ERR_INVALID for a bad descriptor, axis or negative width.
 */
shard_status_t shard_halo_slab_shape(const shard_tile_t* x, int32_t axis, int64_t width, int64_t shape_out[5]);

/*
 * Halo pack (the sending half of the halo exchange, section "PyTorch Dispatch"):
 * copy the `width` interior rows of the tile nearest to `side` (0 = low,
 * 1 = high) along `axis` into the dense slab (shape from shard_halo_slab_shape).
 * `width` is the receiving neighbour's margin on the facing side.
 * Bit-exact copy. width == 0 or an empty slab is a no-op (slab may be NULL).
 * Errors: SHARD_ERR_INVALID (bad descriptor, dtype, axis, side, width < 0, null
 * pointer); SHARD_ERR_UNSUPPORTED when width > ext[axis] (the neighbour would
 * need rows beyond this shard: a multi-hop halo).
 */
shard_status_t shard_halo_pack(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                               int32_t side, int64_t width, void* slab, hipStream_t stream);

/*
 * Halo unpack (the receiving half): write the slab into the margin on
 * (axis, side), whose width is halo_lo[axis] (side 0) or halo_hi[axis] (side 1);
 * the slab shape is shard_halo_slab_shape(x, axis, width). slab == NULL fills
 * the margin with zeros (a global boundary: the convolution's zero padding).
 * Bit-exact copy; a zero-width margin is a no-op.
 * Errors: SHARD_ERR_INVALID (bad descriptor, dtype, axis, side, null tile).
 */
shard_status_t shard_halo_unpack(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                 int32_t side, const void* slab, hipStream_t stream);

/*
 * Both halves of an axis's exchange in one launch each (the faces of an axis are
 * packed together before the sends and its margins filled together after the
 * receives, section "PyTorch Dispatch"): shard_halo_pack_pair equals
 * shard_halo_pack of side 0 with width_lo into slab_lo and of side 1 with
 * width_hi into slab_hi; shard_halo_unpack_pair equals shard_halo_unpack of
 * side 0 from slab_lo and side 1 from slab_hi (NULL: zero-fill that margin).
 * A side of width 0 is skipped. Arguments and errors: as the single calls.
 */
shard_status_t shard_halo_pack_pair(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                                    int64_t width_lo, void* slab_lo, int64_t width_hi, void* slab_hi,
                                    hipStream_t stream);
shard_status_t shard_halo_unpack_pair(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                      const void* slab_lo, const void* slab_hi, hipStream_t stream);

/*
 * Forward convolution over a padded tile:
 *   y[n][j][co] = sum_{ci, t} w[co][ci][t] * tile[n][j*S + t - pad_lo][ci]
 * per axis (j the output row, t the tap), with tile rows outside [0, P_a) read
 * as zero. With the values from shard_conv_geometry this is exactly the shard's
 * slice of the full-domain convolution.
 *   w     [c_out][x->c][kernel0][kernel1][kernel2]  (PyTorch layout), dtype
 *   y     [n][out_ext0][out_ext1][out_ext2][c_out], dtype (overwritten)
 *   ws    device workspace of at least shard_conv_workspace_bytes(0, ...) bytes
 *         (may be NULL when that is 0); contents are scratch.
 * kernel[a] odd in 1..63, stride[a] in 1..64, out_ext[a] >= 0,
 * |pad_lo[a]| < 2^30. Empty output (n or any out_ext 0) is a no-op.
 * Errors: SHARD_ERR_INVALID for malformed arguments (kernel or stride outside
 * 1..64, ...) or a short workspace; SHARD_ERR_UNSUPPORTED for an even kernel
 * (the method's convolutions pad symmetrically, which needs an odd kernel);
 * SHARD_ERR_HIP if a launch fails.
 */
shard_status_t shard_conv_fwd(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* w,
                              int64_t c_out, const int64_t kernel[], const int64_t stride[],
                              const int64_t pad_lo[], const int64_t out_ext[], void* y, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/*
 * shard_conv_fwd for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same convolution and result, bit for bit, without the workspace arguments.
 * Its scratch (the weights rearranged for the matrix instructions) lives in a
 * static device array of the library, 4 MiB, one per GPU, held until the
 * process ends; the call allocates and frees nothing. Every call on a GPU
 * shares that GPU's array, so calls that overlap on one GPU (on different
 * streams, or from different host threads) race and must be serialised by the
 * caller; sequential calls on one stream are safe.
 * Errors: as shard_conv_fwd; SHARD_ERR_UNSUPPORTED also when the workspace
 * shard_conv_fwd would need (shard_conv_workspace_bytes op 0) exceeds 4 MiB;
 * SHARD_ERR_HIP also when the scratch array's address cannot be obtained.
 */
shard_status_t shard_conv_fwd_noalloc(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* w,
                                      int64_t c_out, const int64_t kernel[], const int64_t stride[],
                                      const int64_t pad_lo[], const int64_t out_ext[], void* y,
                                      hipStream_t stream);

/*
 * Received halo slabs for the folded entry points: slab[a][side] is the slab
 * the neighbour on (axis a, side 0 = lo / 1 = hi) sent, laid out as
 * shard_halo_slab_shape(x, a, that margin's width) gives, in the tile's dtype,
 * aligned to the element size (16-byte alignment keeps the fast loads); NULL
 * where the side is a global boundary (zeros).
 * Entries of sides whose margin width is 0 are ignored.
 */
typedef struct {
    const void* slab[3][2];
} shard_halo_src_t;

typedef enum {
    SHARD_REGION_ALL = 0,      /* every owned output */
    SHARD_REGION_INTERIOR = 1, /* outputs whose input rows avoid every margin */
    SHARD_REGION_BOUNDARY = 2  /* the other outputs */
} shard_region_t;

/*
 * The interior outputs of a convolution read off the padded tile: per axis,
 * outputs j in [int_lo[a], int_hi[a]) whose input rows j*S - pad_lo + t,
 * t < kernel[a], all lie in the interior [halo_lo[a], halo_lo[a] + ext[a])
 * (all outputs on an axis without margins). They depend on no halo, so they can
 * be computed while the halo exchange (section "PyTorch Dispatch") is in
 * flight; the paper lists such communication/computation overlap as missing
 * (section "Limitations"). An empty interior has int_lo == int_hi. Host only.
 * Errors: SHARD_ERR_INVALID for malformed arguments.
 */
shard_status_t shard_conv_interior(const shard_tile_t* x, const int64_t kernel[], const int64_t stride[],
                                   const int64_t pad_lo[], const int64_t out_ext[], int64_t int_lo[],
                                   int64_t int_hi[]);

/*
 * shard_conv_fwd with the halo folded into the tile loads: the contents of the
 * tile's margins never affect the result and are never written; the
 * convolution reads each margin voxel from the received slab of its margin
 * (`halo`, NULL = no slabs: every margin zero), a corner voxel from the slab of
 * the later axis. The result equals shard_halo_unpack of every slab in
 * ascending axis order followed by shard_conv_fwd, without the copies into the
 * margins: bit for bit when both calls select the same kernel (margins on one
 * axis, 16-byte aligned slabs) and on integer-valued data, otherwise up to the
 * order of the floating-point sums.
 *   region  SHARD_REGION_ALL, _INTERIOR or _BOUNDARY (shard_region_t): which
 *           outputs are written; the others in y are left untouched. INTERIOR
 *           reads no slab; INTERIOR then BOUNDARY writes what ALL writes.
 * Other arguments, workspace and errors: as shard_conv_fwd (the same workspace
 * size serves every region); SHARD_ERR_INVALID also for an unknown region or a
 * slab not aligned to the element size.
 */
shard_status_t shard_conv_fwd_folded(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                     const shard_halo_src_t* halo, int32_t region, const void* w, int64_t c_out,
                                     const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                     const int64_t out_ext[], void* y, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/*
 * Weight gradient of the shard (its partial; summing the partials of all
 * shards gives the full-domain weight gradient):
 *   dw[co][ci][t] = sum_{n, j} dy[n][j][co] * tile[n][j*S + t - pad_lo][ci]
 * over the shard's outputs j, same tile reading rule as shard_conv_fwd.
 *   dy    [n][out_ext0][out_ext1][out_ext2][c_out], dtype
 *   dw    [c_out][x->c][kernel0][kernel1][kernel2], binary32 (overwritten)
 *   ws    device workspace of at least shard_conv_workspace_bytes(1, ...) bytes.
 *         Its first 32-bit word is the call's device-side status once the call
 *         has completed on the stream: 0 normally; nonzero when a bounded wait
 *         between the waves of a workgroup gave up (possible only if the GPU
 *         stalled a workgroup's waves far beyond any normal schedule), in which
 *         case every dw element is NaN. The caller may read it after
 *         synchronising; the rest of ws is scratch.
 * The summation order is fixed: repeated calls give bit-identical dw.
 * An empty output box writes dw = 0.
 * Errors: as shard_conv_fwd.
 */
shard_status_t shard_conv_wgrad(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* dy,
                                int64_t c_out, const int64_t kernel[], const int64_t stride[],
                                const int64_t pad_lo[], const int64_t out_ext[], float* dw, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/*
 * shard_conv_wgrad with the halo folded into the tile loads, the weight
 * gradient's counterpart of shard_conv_fwd_folded (after a folded forward the
 * margins hold nothing; the received slabs kept from the forward serve the
 * backward pass): the tile's margin rows are never read, each margin voxel
 * comes from the slab of its margin (`halo`, NULL = every margin zero), a
 * corner voxel from the later axis's slab. dw equals shard_halo_unpack of every
 * slab followed by shard_conv_wgrad: bit for bit when both select the same
 * kernel (16-byte aligned slabs; shapes outside the transposed-read kernel
 * for 3x3x3 or 1x3x3 at unit stride with channel counts other than 32 and 64;
 * margins on one axis unless the shape has 16 input channels at unit stride
 * with output channels in blocks of 64; or both calls under
 * SHARD_KERNELS_TILED) and on integer-valued data, otherwise up to the order
 * of the binary32 sums. Other arguments, workspace and errors: as
 * shard_conv_wgrad; SHARD_ERR_INVALID also for a slab not aligned to the
 * element size.
 */
shard_status_t shard_conv_wgrad_folded(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                       const shard_halo_src_t* halo, const void* dy, int64_t c_out,
                                       const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                       const int64_t out_ext[], float* dw, void* ws, size_t ws_bytes,
                                       hipStream_t stream);

/*
 * Input gradient read back onto the padded tile (the backward pass of the
 * shard's convolution; the convolution analogue of the input gradient
 * dL/dx = dL/dz W that the paper writes for a Linear layer, section "What
 * Causes High GPU Memory Usage?", subsection "An Example of Memory Usage"):
 *   dtile[n][p][ci] = sum over co, taps t and outputs j with j*S + t - pad_lo = p
 *                     of w[co][ci][t] * dy[n][j][co]
 * per axis, for every row p of the padded tile, margins included (same tile
 * reading rule as shard_conv_fwd; taps that fall outside the tile drop out).
 * The margin rows then hold gradient that belongs to the neighbours' interiors:
 * shard_halo_pack_margin / shard_halo_accumulate return it, in descending axis
 * order, after which the interior equals the shard's slice of the full-domain
 * input gradient.
 *   x      descriptor of the padded tile (its c is the input channel count Ci)
 *   dy     [n][out_ext0][out_ext1][out_ext2][c_out], dtype
 *   w      [c_out][x->c][kernel0][kernel1][kernel2], dtype (the forward weights)
 *   dtile  the padded tile layout, dtype, every element overwritten (bf16 is
 *          rounded to nearest-even from the binary32 sum; no owned outputs
 *          gives zeros)
 *   ws     device workspace of at least shard_conv_workspace_bytes(2, ...) bytes.
 * Errors: as shard_conv_fwd.
 */
shard_status_t shard_conv_dgrad(const shard_tile_t* x, shard_dtype_t dtype, const void* dy, const void* w,
                                int64_t c_out, const int64_t kernel[], const int64_t stride[],
                                const int64_t pad_lo[], const int64_t out_ext[], void* dtile, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/*
 * Reverse halo, sending half: copy the margin on (axis, side) of a tile holding
 * a gradient (the box shard_halo_unpack writes) into the dense slab
 * (shape shard_halo_slab_shape(x, axis, margin width)), to be returned to the
 * neighbour the margin came from. The halo exchange copies a neighbour's rows
 * into the margin (section "PyTorch Dispatch"); its derivative adds the
 * margin's gradient back onto those rows. Bit-exact copy; a zero-width margin
 * is a no-op. Errors: SHARD_ERR_INVALID (bad descriptor, dtype, axis, side,
 * null pointer).
 */
shard_status_t shard_halo_pack_margin(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                                      int32_t side, void* slab, hipStream_t stream);

/*
 * Reverse halo, receiving half: add the slab to the `width` interior rows on
 * (axis, side) (the box shard_halo_pack reads for that width), element-wise:
 * each sum is formed in binary32 and, for SHARD_BF16, rounded to nearest-even.
 * `width` is the neighbour's margin on the facing side. Axes are returned in
 * descending order (the forward exchange runs ascending), so the slabs of later
 * axes carry the corner gradients into earlier axes' margins, which the earlier
 * axes then return. width == 0 is a no-op.
 * Errors: SHARD_ERR_INVALID (bad descriptor, dtype, axis, side, width < 0, null
 * pointer); SHARD_ERR_UNSUPPORTED when width > ext[axis].
 */
shard_status_t shard_halo_accumulate(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                     int32_t side, int64_t width, const void* slab, hipStream_t stream);

/*
 * Both sides of an axis's reverse exchange in one launch each (the adjoint of
 * shard_halo_pack_pair / shard_halo_unpack_pair): shard_halo_pack_margin_pair
 * equals shard_halo_pack_margin of side 0 into slab_lo and of side 1 into
 * slab_hi (a NULL slab skips that side; a zero-width margin is a no-op);
 * shard_halo_accumulate_pair equals shard_halo_accumulate of side 0 with
 * width_lo from slab_lo followed by side 1 with width_hi from slab_hi (width 0
 * skips a side). When the two faces overlap (width_lo + width_hi > ext[axis])
 * the sides are added by two launches in that order, so the result is the
 * single calls' in every case. Arguments and errors: as the single calls.
 */
shard_status_t shard_halo_pack_margin_pair(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                           int32_t axis, void* slab_lo, void* slab_hi, hipStream_t stream);
shard_status_t shard_halo_accumulate_pair(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                          int64_t width_lo, const void* slab_lo, int64_t width_hi,
                                          const void* slab_hi, hipStream_t stream);

/*
 * Workspace bytes shard_conv_fwd (op 0), shard_conv_wgrad (op 1) or
 * shard_conv_dgrad (op 2) needs for these arguments. A pure function of its
 * arguments (the launch plan does not depend on the device); host only.
 * Returns (size_t)-1 for malformed arguments or an even kernel.
 */
size_t shard_conv_workspace_bytes(int32_t op, const shard_tile_t* x, shard_dtype_t dtype, int64_t c_out,
                                  const int64_t kernel[], const int64_t stride[], const int64_t out_ext[]);

/*
 * Group normalisation of a sharded tensor. A normalisation layer aggregates its
 * statistics across all ranks before normalising (section "PyTorch Dispatch");
 * this library reads it as group normalisation: per batch item n and group g
 * of c / groups consecutive channels, mean and (biased) variance over the
 * group's channels and the whole domain. A shard computes its sums, the sums of
 * all shards are added (the all-reduce), and every shard normalises its
 * interior. Margins are neither read nor written.
 *
 * shard_norm_workspace_bytes: device workspace either call below needs;
 * (size_t)-1 for a bad descriptor, dtype or groups (groups must divide c).
 */
size_t shard_norm_workspace_bytes(const shard_tile_t* x, shard_dtype_t dtype, int64_t groups);

/*
 * The shard's sums over its interior: sums[n][g][0] = sum x, sums[n][g][1] =
 * sum x^2 (float64, device, [x->n][groups][2], overwritten; an empty interior
 * gives zeros). Elements are summed in binary32 within fixed blocks of rows and
 * the blocks in float64, in a fixed order: repeated calls give bit-identical sums.
 * Errors: SHARD_ERR_INVALID (bad descriptor, dtype, groups, null or misaligned
 * pointer, short workspace); SHARD_ERR_HIP if a launch fails.
 */
shard_status_t shard_norm_stats(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int64_t groups,
                                double* sums, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Normalise the interior with the sums of all shards (`sums`, float64 device
 * [x->n][groups][2]) over `count` elements per (n, group) of the whole domain:
 *   mean = S1 / count, var = max(S2 / count - mean^2, 0),
 *   out = (x - mean) / sqrt(var + eps) * gamma[c] + beta[c]
 * evaluated as x * scale[c] + shift[c] with scale and shift formed in float64
 * and rounded once to binary32; gamma and beta are binary32 device arrays of c
 * values. `out` has the tile's layout (interior written, margins untouched)
 * and may be `tile` itself. A bf16 out is rounded to nearest-even.
 * Errors: SHARD_ERR_INVALID (bad descriptor, dtype, groups, count <= 0,
 * eps < 0, null or misaligned pointer, short workspace); SHARD_ERR_HIP.
 */
shard_status_t shard_norm_apply(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const double* sums,
                                double count, double eps, int64_t groups, const float* gamma, const float* beta,
                                void* out, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * One block step of ring attention (section "Performance Benchmarks",
 * subsection "Ring Attention": each device attends its local queries to the
 * key/value block it holds while K and V travel around the ring, accumulating
 * the softmax in log space). Per batch item, head and query row i:
 *   s[i][j]  = scale * q[i] . k[j]              over the block's sk keys
 *   lse_b[i] = log sum_j exp(s[i][j]),  o_b[i] = sum_j exp(s[i][j] - lse_b[i]) v[j]
 * merged into the running state (natural log):
 *   lse[i] <- log(exp(lse[i]) + exp(lse_b[i]))
 *   o[i]   <- exp(old lse[i] - lse[i]) o[i] + exp(lse_b[i] - lse[i]) o_b[i]
 * `first` != 0 starts from the empty state (o = 0, lse = -inf) whatever o and
 * lse hold. After every block of the sequence has been merged, o is
 * softmax(scale q k^T) v over the whole sequence.
 *   q      [batch][heads][sq][head_dim], dtype SHARD_BF16
 *   k, v   [batch][heads][sk][head_dim], SHARD_BF16 (sk = 0: an empty block)
 *   o      [batch][heads][sq][head_dim], binary32, read (unless first) and written
 *   lse    [batch][heads][sq], binary32, read (unless first) and written
 * head_dim 64 or 128; q, k, v and o 16-byte aligned; sk * head_dim * 2 < 2^32.
 * Scores and sums are binary32; the probabilities enter the second product
 * rounded to bf16 (to nearest even).
 * Errors: SHARD_ERR_UNSUPPORTED for another dtype or head_dim or sizes past the
 * limits; SHARD_ERR_INVALID for negative sizes, null or misaligned buffers, a
 * non-finite scale; SHARD_ERR_HIP if a launch fails.
 */
shard_status_t shard_attn_block(int64_t batch, int64_t heads, int64_t sq, int64_t sk, int64_t head_dim,
                                shard_dtype_t dtype, float scale, const void* q, const void* k, const void* v,
                                float* o, float* lse, int32_t first, hipStream_t stream);

/* Static, human-readable text for a status code. Never NULL. */
const char* shard_status_string(shard_status_t status);

/*
 * Options of the calling host thread, applied to its later calls (other
 * threads keep their own; a new thread starts from the defaults):
 *   kernels     which kernel family the convolutions (fwd, wgrad, dgrad and
 *               the folded calls) take: SHARD_KERNELS_FASTEST (default) the
 *               fastest applicable one, SHARD_KERNELS_TILED the general tiled
 *               MFMA kernels (no shape-specialised kernel), SHARD_KERNELS_DIRECT
 *               the plain direct kernels. All compute the same function; the
 *               families exist to cross-check one another (the MFMA families
 *               agree bit for bit on integer-valued data).
 *   wait_polls  the poll bound of the weight gradient's hand-off waits between
 *               the waves of a workgroup; 0 keeps the default (2^20 polls).
 *               A small bound makes the waits give up, which the status word
 *               of shard_conv_wgrad reports: the way to check that report.
 * opts == NULL restores the defaults.
 * Errors: SHARD_ERR_INVALID for an unknown kernel family.
 */
typedef enum { SHARD_KERNELS_FASTEST = 0, SHARD_KERNELS_TILED = 1, SHARD_KERNELS_DIRECT = 2 } shard_kernels_t;
typedef struct {
    int32_t kernels;
    uint32_t wait_polls;
} shard_call_opts_t;
shard_status_t shard_set_call_opts(const shard_call_opts_t* opts);

#ifdef __cplusplus
}
#endif

#endif /* SHARDCONV_H */
