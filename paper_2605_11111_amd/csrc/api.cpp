// C-ABI entry points: argument validation on the host (before any launch, so
// an error writes nothing), normalisation to three spatial axes, dispatch.
#include <algorithm>
#include <cmath>

#include "attention.h"
#include "internal.h"

namespace shardconv {

namespace {
// per host thread: calls from other threads never see another thread's options
thread_local CallOpts tl_opts{SHARD_KERNELS_FASTEST, 0u};
}  // namespace

const CallOpts& call_opts() { return tl_opts; }
bool force_generic() { return tl_opts.kernels == SHARD_KERNELS_DIRECT; }
bool force_tiled() { return tl_opts.kernels == SHARD_KERNELS_TILED; }

size_t generic_wgrad_workspace(const Tile3& t, const Conv3& cv);
hipError_t generic_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                              float* dw, void* ws, const Fold* fold, hipStream_t s);

}  // namespace shardconv

using namespace shardconv;

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 40;

bool valid_dtype(shard_dtype_t d) { return d == SHARD_F32 || d == SHARD_BF16; }
int esize(shard_dtype_t d) { return d == SHARD_F32 ? 4 : 2; }
bool aligned(const void* p, int a) { return (reinterpret_cast<uintptr_t>(p) % uintptr_t(a)) == 0; }

// Product of non-negative sizes with an overflow guard (false if >= 2^62).
bool safe_mul(int64_t& acc, int64_t v)
{
    if (v == 0) {
        acc = 0;
        return true;
    }
    if (acc > (int64_t(1) << 62) / v) return false;
    acc *= v;
    return true;
}

bool norm_tile(const shard_tile_t* x, shard_dtype_t dt, Tile3& t)
{
    if (!x || x->ndim < 1 || x->ndim > 3 || !valid_dtype(dt)) return false;
    if (x->n < 0 || x->n > kMaxDim || x->c < 1 || x->c > kMaxDim) return false;
    t.n = x->n;
    t.c = x->c;
    t.esz = esize(dt);
    const int off = 3 - x->ndim;
    for (int k = 0; k < 3; ++k) {
        t.lo[k] = t.hi[k] = 0;
        t.ext[k] = 1;
    }
    for (int a = 0; a < x->ndim; ++a) {
        const int k = off + a;
        if (x->ext[a] < 0 || x->halo_lo[a] < 0 || x->halo_hi[a] < 0) return false;
        if (x->ext[a] > kMaxDim || x->halo_lo[a] > kMaxDim || x->halo_hi[a] > kMaxDim) return false;
        t.lo[k] = x->halo_lo[a];
        t.ext[k] = x->ext[a];
        t.hi[k] = x->halo_hi[a];
    }
    int64_t total = t.n;
    for (int k = 0; k < 3; ++k) {
        t.P[k] = t.lo[k] + t.ext[k] + t.hi[k];
        if (!safe_mul(total, t.P[k])) return false;
    }
    int64_t bytes = total;
    return safe_mul(bytes, t.c * t.esz);
}

int64_t tile_elems(const Tile3& t) { return t.n * t.P[0] * t.P[1] * t.P[2] * t.c; }

bool norm_conv(const shard_tile_t* x, const Tile3& t, int64_t c_out, const int64_t kernel[], const int64_t stride[],
               const int64_t pad_lo[], const int64_t out_ext[], Conv3& cv)
{
    if (c_out < 1 || c_out > kMaxDim || !kernel || !stride || !out_ext) return false;
    const int off = 3 - x->ndim;
    cv.cout = c_out;
    for (int k = 0; k < 3; ++k) {
        cv.K[k] = 1;
        cv.S[k] = 1;
        cv.pad[k] = 0;
        cv.O[k] = 1;
    }
    for (int a = 0; a < x->ndim; ++a) {
        const int k = off + a;
        if (kernel[a] < 1 || kernel[a] > 64 || stride[a] < 1 || stride[a] > 64) return false;
        if (out_ext[a] < 0 || out_ext[a] > kMaxDim) return false;
        const int64_t p = pad_lo ? pad_lo[a] : 0;
        if (p <= -(int64_t(1) << 30) || p >= (int64_t(1) << 30)) return false;
        cv.K[k] = kernel[a];
        cv.S[k] = stride[a];
        cv.pad[k] = p;
        cv.O[k] = out_ext[a];
    }
    int64_t total = t.n;
    for (int k = 0; k < 3; ++k)
        if (!safe_mul(total, cv.O[k])) return false;
    int64_t wsz = cv.cout;
    if (!safe_mul(wsz, t.c) || !safe_mul(wsz, cv.taps())) return false;
    return safe_mul(total, cv.cout);
}

// The convolutions this library implements pad symmetrically ("same"
// padding, P = (K - 1) / 2 per side), which needs an odd kernel on every axis.
bool odd_kernel(const shard_tile_t* x, const int64_t kernel[])
{
    for (int a = 0; a < x->ndim; ++a)
        if (kernel[a] % 2 == 0) return false;
    return true;
}

// The box a slab covers on internal axis k: rows [r0, r1) on k, the padded
// extent on earlier axes, the interior on later ones.
void slab_spans(const Tile3& t, int k, int64_t r0, int64_t r1, int64_t start[3], int64_t cnt[3])
{
    for (int b = 0; b < 3; ++b) {
        if (b < k) {
            start[b] = 0;
            cnt[b] = t.P[b];
        } else if (b == k) {
            start[b] = r0;
            cnt[b] = r1 - r0;
        } else {
            start[b] = t.lo[b];
            cnt[b] = t.ext[b];
        }
    }
}

BoxCopy make_box(const Tile3& t, int k, int64_t r0, int64_t r1)
{
    int64_t start[3], cnt[3];
    slab_spans(t, k, r0, r1, start, cnt);
    const int64_t es = t.esz;
    // dims outermost first: n, axis0, axis1, axis2; byte strides in the tile
    int64_t dcnt[4] = {t.n, cnt[0], cnt[1], cnt[2]};
    int64_t dstr[4] = {t.P[0] * t.P[1] * t.P[2] * t.c * es, t.P[1] * t.P[2] * t.c * es, t.P[2] * t.c * es, t.c * es};
    int64_t full[4] = {t.n, t.P[0], t.P[1], t.P[2]};
    BoxCopy b{};
    b.base = ((start[0] * t.P[1] + start[1]) * t.P[2] + start[2]) * t.c * es;
    // merge contiguous inner dims into the run
    int64_t run = t.c * es;
    int d = 3;
    run *= dcnt[d];  // axis 2 rows are always contiguous
    --d;
    while (d >= 0 && dcnt[d + 1] == full[d + 1] && dstr[d] == run) {
        run *= dcnt[d];
        --d;
    }
    b.run = run;
    // remaining outer dims 0..d (at most 3), right-aligned into cnt[3]
    for (int i = 0; i < 3; ++i) {
        b.cnt[i] = 1;
        b.tstride[i] = 0;
    }
    for (int i = d, j = 2; i >= 0; --i, --j) {
        b.cnt[j] = dcnt[i];
        b.tstride[j] = dstr[i];
    }
    return b;
}

shard_status_t map_hip(hipError_t e) { return e == hipSuccess ? SHARD_OK : SHARD_ERR_HIP; }

// A weight gradient over no outputs: dw = 0 (the direct kernel's empty sum) and
// a cleared status word.
hipError_t empty_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, float* dw, void* ws, hipStream_t s)
{
    hipError_t e = launch_wgrad_status_clear(static_cast<uint32_t*>(ws), s);
    if (e != hipSuccess) return e;
    return generic_conv_wgrad(t, cv, dt, nullptr, nullptr, dw, static_cast<char*>(ws) + kWgradStatusBytes, nullptr, s);
}

// The Fold of a call: every axis with a margin reads it from the received slab
// (null: zero). False for a slab not aligned to the element size.
bool make_fold(const shard_tile_t* x, const Tile3& t, const shard_halo_src_t* halo, Fold& f)
{
    f = Fold{};
    const int off = 3 - x->ndim;
    for (int k = 0; k < 3; ++k) {
        f.lo[k] = t.lo[k];
        f.ext[k] = t.ext[k];
        f.P[k] = t.P[k];
        if (t.lo[k] > 0 || t.hi[k] > 0) f.mask |= 1u << k;
        for (int sd = 0; sd < 2; ++sd) {
            const int64_t width = sd == 0 ? t.lo[k] : t.hi[k];
            const void* p = (halo && k >= off && width > 0) ? halo->slab[k - off][sd] : nullptr;
            if (!aligned(p, t.esz)) return false;
            f.slab[k][sd] = static_cast<const char*>(p);
        }
    }
    return true;
}

// Interior outputs per internal axis: [jlo, jhi) of the outputs whose input rows
// j*S - pad + t (t < K) lie in [lo, lo + ext); every output on an axis without
// margins. jhi >= jlo.
void interior_box(const Tile3& t, const Conv3& cv, int64_t jlo[3], int64_t jhi[3])
{
    for (int k = 0; k < 3; ++k) {
        jlo[k] = 0;
        jhi[k] = cv.O[k];
        if (t.lo[k] > 0) {
            const int64_t a = t.lo[k] + cv.pad[k];  // first j with j*S - pad >= lo
            jlo[k] = a <= 0 ? 0 : std::min(cv.O[k], ceil_div(a, cv.S[k]));
        }
        if (t.hi[k] > 0) {
            const int64_t b = t.lo[k] + t.ext[k] - cv.K[k] + cv.pad[k];  // last j has j*S <= b
            jhi[k] = b < 0 ? 0 : std::min(cv.O[k], b / cv.S[k] + 1);
        }
        if (jhi[k] < jlo[k]) jhi[k] = jlo[k];
    }
}

// The output boxes of a region: ALL is the owned box, INTERIOR the interior box,
// BOUNDARY the owned box minus the interior, peeled axis by axis (axis k's two
// slabs span the interior on earlier axes and everything on later ones).
int region_boxes(const Tile3& t, const Conv3& cv, int32_t region, Region out[6])
{
    int nb = 0;
    int64_t jlo[3], jhi[3];
    interior_box(t, cv, jlo, jhi);
    if (region == SHARD_REGION_ALL || region == SHARD_REGION_INTERIOR) {
        Region r{};
        for (int k = 0; k < 3; ++k) {
            r.org[k] = region == SHARD_REGION_ALL ? 0 : jlo[k];
            r.ext[k] = region == SHARD_REGION_ALL ? cv.O[k] : jhi[k] - jlo[k];
        }
        out[nb++] = r;
        return nb;
    }
    for (int k = 0; k < 3; ++k) {
        for (int sd = 0; sd < 2; ++sd) {
            Region r{};
            for (int b = 0; b < 3; ++b) {
                if (b < k) {
                    r.org[b] = jlo[b];
                    r.ext[b] = jhi[b] - jlo[b];
                } else if (b > k) {
                    r.org[b] = 0;
                    r.ext[b] = cv.O[b];
                }
            }
            r.org[k] = sd == 0 ? 0 : jhi[k];
            r.ext[k] = sd == 0 ? jlo[k] : cv.O[k] - jhi[k];
            if (r.ext[0] * r.ext[1] * r.ext[2] > 0) out[nb++] = r;
        }
    }
    return nb;
}

}  // namespace

extern "C" {

shard_status_t shard_set_call_opts(const shard_call_opts_t* opts)
{
    if (!opts) {
        tl_opts = CallOpts{SHARD_KERNELS_FASTEST, 0u};
        return SHARD_OK;
    }
    if (opts->kernels != SHARD_KERNELS_FASTEST && opts->kernels != SHARD_KERNELS_TILED &&
        opts->kernels != SHARD_KERNELS_DIRECT)
        return SHARD_ERR_INVALID;
    tl_opts = CallOpts{opts->kernels, opts->wait_polls};
    return SHARD_OK;
}

const char* shard_status_string(shard_status_t s)
{
    switch (s) {
    case SHARD_OK:
        return "ok";
    case SHARD_ERR_INVALID:
        return "invalid argument";
    case SHARD_ERR_UNSUPPORTED:
        return "unsupported argument";
    case SHARD_ERR_HIP:
        return "HIP runtime error";
    default:
        return "unknown status";
    }
}

shard_status_t shard_halo_slab_shape(const shard_tile_t* x, int32_t axis, int64_t width, int64_t shape_out[5])
{
    Tile3 t;
    if (!shape_out || !norm_tile(x, SHARD_F32, t) || axis < 0 || axis >= x->ndim || width < 0 || width > kMaxDim)
        return SHARD_ERR_INVALID;
    shape_out[0] = x->n;
    for (int b = 0; b < 3; ++b) {
        if (b >= x->ndim)
            shape_out[1 + b] = 1;
        else if (b < axis)
            shape_out[1 + b] = x->halo_lo[b] + x->ext[b] + x->halo_hi[b];
        else if (b == axis)
            shape_out[1 + b] = width;
        else
            shape_out[1 + b] = x->ext[b];
    }
    shape_out[4] = x->c;
    return SHARD_OK;
}

shard_status_t shard_halo_pack(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                               int32_t side, int64_t width, void* slab, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || (side != 0 && side != 1) || width < 0)
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    if (width > t.ext[k]) return SHARD_ERR_UNSUPPORTED;
    const int64_t r0 = side == 0 ? t.lo[k] : t.lo[k] + t.ext[k] - width;
    int64_t start[3], cnt[3];
    slab_spans(t, k, r0, r0 + width, start, cnt);
    if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) return SHARD_OK;
    if (!tile || !slab || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
    return map_hip(launch_box_copy(make_box(t, k, r0, r0 + width), TILE_TO_SLAB, tile, slab, stream));
}

shard_status_t shard_halo_unpack(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                 int32_t side, const void* slab, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || (side != 0 && side != 1))
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    const int64_t r0 = side == 0 ? 0 : t.lo[k] + t.ext[k];
    const int64_t r1 = side == 0 ? t.lo[k] : t.P[k];
    int64_t start[3], cnt[3];
    slab_spans(t, k, r0, r1, start, cnt);
    if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) return SHARD_OK;
    if (!tile || !aligned(tile, t.esz) || (slab && !aligned(slab, t.esz))) return SHARD_ERR_INVALID;
    const BoxCopy b = make_box(t, k, r0, r1);
    if (!slab) return map_hip(launch_box_copy(b, ZERO_TILE, nullptr, tile, stream));
    return map_hip(launch_box_copy(b, SLAB_TO_TILE, slab, tile, stream));
}

shard_status_t shard_halo_pack_pair(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                                    int64_t width_lo, void* slab_lo, int64_t width_hi, void* slab_hi,
                                    hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || width_lo < 0 || width_hi < 0)
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    if (width_lo > t.ext[k] || width_hi > t.ext[k]) return SHARD_ERR_UNSUPPORTED;
    BoxCopy boxes[2];
    const BoxCopy* bp[2];
    CopyDir dirs[2] = {TILE_TO_SLAB, TILE_TO_SLAB};
    const void* srcs[2] = {tile, tile};
    void* dsts[2];
    int n = 0;
    for (int sd = 0; sd < 2; ++sd) {
        const int64_t width = sd == 0 ? width_lo : width_hi;
        void* slab = sd == 0 ? slab_lo : slab_hi;
        const int64_t r0 = sd == 0 ? t.lo[k] : t.lo[k] + t.ext[k] - width;
        int64_t start[3], cnt[3];
        slab_spans(t, k, r0, r0 + width, start, cnt);
        if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) continue;
        if (!tile || !slab || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
        boxes[n] = make_box(t, k, r0, r0 + width);
        bp[n] = &boxes[n];
        dsts[n] = slab;
        ++n;
    }
    if (n == 0) return SHARD_OK;
    return map_hip(launch_box_copies(bp, dirs, srcs, dsts, n, stream));
}

shard_status_t shard_halo_unpack_pair(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                      const void* slab_lo, const void* slab_hi, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim) return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    BoxCopy boxes[2];
    const BoxCopy* bp[2];
    CopyDir dirs[2];
    const void* srcs[2];
    void* dsts[2] = {tile, tile};
    int n = 0;
    for (int sd = 0; sd < 2; ++sd) {
        const void* slab = sd == 0 ? slab_lo : slab_hi;
        const int64_t r0 = sd == 0 ? 0 : t.lo[k] + t.ext[k];
        const int64_t r1 = sd == 0 ? t.lo[k] : t.P[k];
        int64_t start[3], cnt[3];
        slab_spans(t, k, r0, r1, start, cnt);
        if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) continue;
        if (!tile || !aligned(tile, t.esz) || (slab && !aligned(slab, t.esz))) return SHARD_ERR_INVALID;
        boxes[n] = make_box(t, k, r0, r1);
        bp[n] = &boxes[n];
        dirs[n] = slab ? SLAB_TO_TILE : ZERO_TILE;
        srcs[n] = slab;
        ++n;
    }
    if (n == 0) return SHARD_OK;
    return map_hip(launch_box_copies(bp, dirs, srcs, dsts, n, stream));
}

shard_status_t shard_halo_pack_margin(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int32_t axis,
                                      int32_t side, void* slab, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || (side != 0 && side != 1))
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    const int64_t r0 = side == 0 ? 0 : t.lo[k] + t.ext[k];
    const int64_t r1 = side == 0 ? t.lo[k] : t.P[k];
    int64_t start[3], cnt[3];
    slab_spans(t, k, r0, r1, start, cnt);
    if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) return SHARD_OK;
    if (!tile || !slab || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
    return map_hip(launch_box_copy(make_box(t, k, r0, r1), TILE_TO_SLAB, tile, slab, stream));
}

shard_status_t shard_halo_accumulate(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                     int32_t side, int64_t width, const void* slab, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || (side != 0 && side != 1) || width < 0)
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    if (width > t.ext[k]) return SHARD_ERR_UNSUPPORTED;
    const int64_t r0 = side == 0 ? t.lo[k] : t.lo[k] + t.ext[k] - width;
    int64_t start[3], cnt[3];
    slab_spans(t, k, r0, r0 + width, start, cnt);
    if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) return SHARD_OK;
    if (!tile || !slab || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
    return map_hip(launch_box_add(make_box(t, k, r0, r0 + width), t.esz, slab, tile, stream));
}

shard_status_t shard_halo_pack_margin_pair(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                           int32_t axis, void* slab_lo, void* slab_hi, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim) return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    BoxCopy boxes[2];
    const BoxCopy* bp[2];
    CopyDir dirs[2] = {TILE_TO_SLAB, TILE_TO_SLAB};
    const void* srcs[2] = {tile, tile};
    void* dsts[2];
    int n = 0;
    for (int sd = 0; sd < 2; ++sd) {
        void* slab = sd == 0 ? slab_lo : slab_hi;
        if (!slab) continue;
        const int64_t r0 = sd == 0 ? 0 : t.lo[k] + t.ext[k];
        const int64_t r1 = sd == 0 ? t.lo[k] : t.P[k];
        int64_t start[3], cnt[3];
        slab_spans(t, k, r0, r1, start, cnt);
        if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) continue;
        if (!tile || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
        boxes[n] = make_box(t, k, r0, r1);
        bp[n] = &boxes[n];
        dsts[n] = slab;
        ++n;
    }
    if (n == 0) return SHARD_OK;
    return map_hip(launch_box_copies(bp, dirs, srcs, dsts, n, stream));
}

shard_status_t shard_halo_accumulate_pair(const shard_tile_t* x, shard_dtype_t dtype, void* tile, int32_t axis,
                                          int64_t width_lo, const void* slab_lo, int64_t width_hi,
                                          const void* slab_hi, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || axis < 0 || axis >= x->ndim || width_lo < 0 || width_hi < 0)
        return SHARD_ERR_INVALID;
    const int k = 3 - x->ndim + axis;
    if (width_lo > t.ext[k] || width_hi > t.ext[k]) return SHARD_ERR_UNSUPPORTED;
    BoxCopy boxes[2];
    const BoxCopy* bp[2];
    const void* slabs[2];
    int n = 0;
    for (int sd = 0; sd < 2; ++sd) {
        const int64_t width = sd == 0 ? width_lo : width_hi;
        const void* slab = sd == 0 ? slab_lo : slab_hi;
        const int64_t r0 = sd == 0 ? t.lo[k] : t.lo[k] + t.ext[k] - width;
        int64_t start[3], cnt[3];
        slab_spans(t, k, r0, r0 + width, start, cnt);
        if (t.n * cnt[0] * cnt[1] * cnt[2] == 0) continue;
        if (!tile || !slab || !aligned(tile, t.esz) || !aligned(slab, t.esz)) return SHARD_ERR_INVALID;
        boxes[n] = make_box(t, k, r0, r0 + width);
        bp[n] = &boxes[n];
        slabs[n] = slab;
        ++n;
    }
    if (n == 0) return SHARD_OK;
    if (n == 2 && width_lo + width_hi > t.ext[k]) {
        // overlapping faces: one launch per side, in order
        hipError_t e = launch_box_adds(bp, t.esz, slabs, tile, 1, stream);
        if (e != hipSuccess) return map_hip(e);
        return map_hip(launch_box_adds(bp + 1, t.esz, slabs + 1, tile, 1, stream));
    }
    return map_hip(launch_box_adds(bp, t.esz, slabs, tile, n, stream));
}

size_t shard_conv_workspace_bytes(int32_t op, const shard_tile_t* x, shard_dtype_t dtype, int64_t c_out,
                                  const int64_t kernel[], const int64_t stride[], const int64_t out_ext[])
{
    Tile3 t;
    Conv3 cv;
    if (op < 0 || op > 2 || !norm_tile(x, dtype, t) || !norm_conv(x, t, c_out, kernel, stride, nullptr, out_ext, cv) ||
        !odd_kernel(x, kernel))
        return size_t(-1);
    if (op == 0) return conv_fwd_workspace(t, cv, dtype);
    if (op == 1) return conv_wgrad_workspace(t, cv, dtype);
    return conv_dgrad_workspace(t, cv, dtype);
}

shard_status_t shard_conv_fwd(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* w,
                              int64_t c_out, const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                              const int64_t out_ext[], void* y, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    if (t.n * cv.out_voxels() == 0) return SHARD_OK;
    const size_t need = conv_fwd_workspace(t, cv, dtype);
    if (ws_bytes < need || (need > 0 && !ws)) return SHARD_ERR_INVALID;
    if ((tile_elems(t) > 0 && !tile) || !w || !y) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(w, t.esz) || !aligned(y, t.esz) || !aligned(ws, 16))
        return SHARD_ERR_INVALID;
    return map_hip(launch_conv_fwd(t, cv, dtype, tile, w, y, ws, stream));
}

shard_status_t shard_conv_fwd_noalloc(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* w,
                                      int64_t c_out, const int64_t kernel[], const int64_t stride[],
                                      const int64_t pad_lo[], const int64_t out_ext[], void* y, hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    if (t.n * cv.out_voxels() == 0) return SHARD_OK;
    if (conv_fwd_workspace(t, cv, dtype) > conv_fwd_noalloc_limit()) return SHARD_ERR_UNSUPPORTED;
    if ((tile_elems(t) > 0 && !tile) || !w || !y) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(w, t.esz) || !aligned(y, t.esz)) return SHARD_ERR_INVALID;
    return map_hip(launch_conv_fwd_noalloc(t, cv, dtype, tile, w, y, stream));
}

shard_status_t shard_conv_interior(const shard_tile_t* x, const int64_t kernel[], const int64_t stride[],
                                   const int64_t pad_lo[], const int64_t out_ext[], int64_t int_lo[],
                                   int64_t int_hi[])
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, SHARD_F32, t) || !pad_lo || !int_lo || !int_hi ||
        !norm_conv(x, t, 1, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    int64_t jlo[3], jhi[3];
    interior_box(t, cv, jlo, jhi);
    const int off = 3 - x->ndim;
    for (int a = 0; a < x->ndim; ++a) {
        int_lo[a] = jlo[off + a];
        int_hi[a] = jhi[off + a];
    }
    return SHARD_OK;
}

shard_status_t shard_conv_fwd_folded(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                     const shard_halo_src_t* halo, int32_t region, const void* w, int64_t c_out,
                                     const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                     const int64_t out_ext[], void* y, void* ws, size_t ws_bytes,
                                     hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    if (region != SHARD_REGION_ALL && region != SHARD_REGION_INTERIOR && region != SHARD_REGION_BOUNDARY)
        return SHARD_ERR_INVALID;
    if (t.n * cv.out_voxels() == 0) return SHARD_OK;
    const size_t need = conv_fwd_workspace(t, cv, dtype);
    if (ws_bytes < need || (need > 0 && !ws)) return SHARD_ERR_INVALID;
    if ((tile_elems(t) > 0 && !tile) || !w || !y) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(w, t.esz) || !aligned(y, t.esz) || !aligned(ws, 16))
        return SHARD_ERR_INVALID;
    Fold f;
    if (!make_fold(x, t, halo, f)) return SHARD_ERR_INVALID;
    const OutMap om = dense_out(cv);
    const Fold* fold = f.mask ? &f : nullptr;
    const FwdFamily fam = fwd_family(t, cv, dtype, tile, y, om, fold, ws);
    // The interior outputs read no margin, so the plain kernels serve them (rows
    // a brick stages past the region feed only outputs that are not written).
    // On the W-march kernel the folded loads cost more than a separate launch
    // over the boundary, so the whole box runs as interior + boundary there.
    Region boxes[7];
    bool folded[7];
    int nb = 0;
    if (region == SHARD_REGION_ALL && fold && fam == FWD_ROWS) {
        nb = region_boxes(t, cv, SHARD_REGION_INTERIOR, boxes);
        for (int i = 0; i < nb; ++i) folded[i] = false;
        const int nbb = region_boxes(t, cv, SHARD_REGION_BOUNDARY, boxes + nb);
        for (int i = nb; i < nb + nbb; ++i) folded[i] = true;
        nb += nbb;
    } else {
        nb = region_boxes(t, cv, region, boxes);
        for (int i = 0; i < nb; ++i) folded[i] = fold && region != SHARD_REGION_INTERIOR;
    }
    bool laid = false;  // weight fragments in ws (the first non-empty region lays them out)
    auto nonempty = [&](const Region& r) { return t.n * r.ext[0] * r.ext[1] * r.ext[2] > 0; };
    for (int i = 0; i < nb; ++i) {
        // two regions of the W-march kernel that differ along axis 0 only (the
        // boundary planes of a tile sharded along axis 0), or up to four
        // regions of the tiled kernel (boundary slabs, too thin to fill the
        // part one by one), go in one launch
        if (fam == FWD_TILED) {
            int run = 0;  // consecutive non-empty regions with the same folding
            while (i + run < nb && run < 4 && folded[i + run] == folded[i] && nonempty(boxes[i + run])) ++run;
            bool done = false;
            for (int k = run; k >= 2 && !done; --k) {
                const hipError_t e = launch_conv_fwd_tiled_group(t, cv, dtype, tile, w, y, om, boxes + i, k,
                                                                 folded[i] ? fold : nullptr, ws, stream, laid);
                if (e == hipSuccess) {
                    laid = true;
                    i += k - 1;
                    done = true;
                } else if (e != hipErrorNotSupported) {
                    return SHARD_ERR_HIP;
                }
            }
            if (done) continue;
        }
        if (fam == FWD_ROWS && i + 1 < nb && folded[i] == folded[i + 1] && nonempty(boxes[i]) &&
            nonempty(boxes[i + 1])) {
            const Fold* fi = folded[i] ? fold : nullptr;
            const hipError_t e =
                launch_conv_fwd_region_pair(t, cv, dtype, tile, w, y, boxes[i], boxes[i + 1], fi, ws, stream, laid);
            if (e == hipSuccess) {
                laid = true;
                ++i;
                continue;
            }
            if (e != hipErrorNotSupported) return SHARD_ERR_HIP;
        }
        const hipError_t e = launch_conv_fwd_region(t, cv, dtype, tile, w, y, om, boxes[i], folded[i] ? fold : nullptr,
                                                    fam, ws, stream, laid);
        if (e != hipSuccess) return SHARD_ERR_HIP;
        laid = laid || nonempty(boxes[i]);
    }
    return SHARD_OK;
}

shard_status_t shard_attn_block(int64_t batch, int64_t heads, int64_t sq, int64_t sk, int64_t head_dim,
                                shard_dtype_t dtype, float scale, const void* q, const void* k, const void* v,
                                float* o, float* lse, int32_t first, hipStream_t stream)
{
    if (batch < 0 || heads < 0 || sq < 0 || sk < 0 || head_dim < 1 || !valid_dtype(dtype) || !std::isfinite(scale))
        return SHARD_ERR_INVALID;
    if (dtype != SHARD_BF16 || (head_dim != 64 && head_dim != 128)) return SHARD_ERR_UNSUPPORTED;
    if (batch > kMaxDim || heads > kMaxDim || sq > kMaxDim || sk > kMaxDim) return SHARD_ERR_UNSUPPORTED;
    int64_t bh = batch;
    if (!safe_mul(bh, heads)) return SHARD_ERR_UNSUPPORTED;
    if (bh * sq == 0) return SHARD_OK;
    if (!q || !o || !lse || !aligned(q, 16) || !aligned(o, 16) || !aligned(lse, 4)) return SHARD_ERR_INVALID;
    if (sk > 0 && (!k || !v || !aligned(k, 16) || !aligned(v, 16))) return SHARD_ERR_INVALID;
    const hipError_t e = launch_attn_block(bh, sq, sk, head_dim, scale, q, k ? k : q, v ? v : q, o, lse, first != 0,
                                           stream);
    if (e == hipErrorNotSupported) return SHARD_ERR_UNSUPPORTED;
    return map_hip(e);
}

shard_status_t shard_conv_wgrad(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const void* dy,
                                int64_t c_out, const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                const int64_t out_ext[], float* dw, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    const size_t need = conv_wgrad_workspace(t, cv, dtype);
    if (ws_bytes < need || (need > 0 && !ws)) return SHARD_ERR_INVALID;
    if (!dw || !aligned(dw, 4) || !aligned(ws, 16)) return SHARD_ERR_INVALID;
    const bool empty = t.n * cv.out_voxels() == 0;
    if (!empty && ((tile_elems(t) > 0 && !tile) || !dy)) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(dy, t.esz)) return SHARD_ERR_INVALID;
    if (empty) return map_hip(empty_wgrad(t, cv, dtype, dw, ws, stream));
    return map_hip(launch_conv_wgrad(t, cv, dtype, tile, dy, dw, ws, stream));
}

shard_status_t shard_conv_wgrad_folded(const shard_tile_t* x, shard_dtype_t dtype, const void* tile,
                                       const shard_halo_src_t* halo, const void* dy, int64_t c_out,
                                       const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                       const int64_t out_ext[], float* dw, void* ws, size_t ws_bytes,
                                       hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    const size_t need = conv_wgrad_workspace(t, cv, dtype);
    if (ws_bytes < need || (need > 0 && !ws)) return SHARD_ERR_INVALID;
    if (!dw || !aligned(dw, 4) || !aligned(ws, 16)) return SHARD_ERR_INVALID;
    const bool empty = t.n * cv.out_voxels() == 0;
    if (!empty && ((tile_elems(t) > 0 && !tile) || !dy)) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(dy, t.esz)) return SHARD_ERR_INVALID;
    Fold f;
    if (!make_fold(x, t, halo, f)) return SHARD_ERR_INVALID;
    if (empty) return map_hip(empty_wgrad(t, cv, dtype, dw, ws, stream));
    if (!f.mask) return map_hip(launch_conv_wgrad(t, cv, dtype, tile, dy, dw, ws, stream));
    return map_hip(launch_conv_wgrad_folded(t, cv, dtype, tile, dy, dw, ws, f, stream));
}

shard_status_t shard_conv_dgrad(const shard_tile_t* x, shard_dtype_t dtype, const void* dy, const void* w,
                                int64_t c_out, const int64_t kernel[], const int64_t stride[], const int64_t pad_lo[],
                                const int64_t out_ext[], void* dtile, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Tile3 t;
    Conv3 cv;
    if (!norm_tile(x, dtype, t) || !pad_lo || !norm_conv(x, t, c_out, kernel, stride, pad_lo, out_ext, cv))
        return SHARD_ERR_INVALID;
    if (!odd_kernel(x, kernel)) return SHARD_ERR_UNSUPPORTED;
    if (tile_elems(t) == 0) return SHARD_OK;
    const size_t need = conv_dgrad_workspace(t, cv, dtype);
    if (ws_bytes < need || (need > 0 && !ws)) return SHARD_ERR_INVALID;
    if (!dtile || !w || !aligned(dtile, t.esz) || !aligned(w, t.esz) || !aligned(dy, t.esz) || !aligned(ws, 16))
        return SHARD_ERR_INVALID;
    if (t.n * cv.out_voxels() == 0) {
        // no owned outputs: the tile's gradient is zero
        BoxCopy b{};
        b.base = 0;
        b.run = tile_elems(t) * t.esz;
        for (int i = 0; i < 3; ++i) {
            b.cnt[i] = 1;
            b.tstride[i] = 0;
        }
        return map_hip(launch_box_copy(b, ZERO_TILE, nullptr, dtile, stream));
    }
    if (!dy) return SHARD_ERR_INVALID;
    return map_hip(launch_conv_dgrad(t, cv, dtype, dy, w, dtile, ws, stream));
}

size_t shard_norm_workspace_bytes(const shard_tile_t* x, shard_dtype_t dtype, int64_t groups)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || groups < 1 || groups > t.c || t.c % groups != 0) return size_t(-1);
    return norm_workspace(t, groups);
}

shard_status_t shard_norm_stats(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, int64_t groups,
                                double* sums, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || groups < 1 || groups > t.c || t.c % groups != 0) return SHARD_ERR_INVALID;
    if (t.n == 0) return SHARD_OK;
    const size_t need = norm_workspace(t, groups);
    if (!sums || !ws || ws_bytes < need || !aligned(sums, 8) || !aligned(ws, 16)) return SHARD_ERR_INVALID;
    if (tile_elems(t) > 0 && (!tile || !aligned(tile, t.esz))) return SHARD_ERR_INVALID;
    return map_hip(launch_norm_stats(t, dtype, tile, groups, sums, ws, stream));
}

shard_status_t shard_norm_apply(const shard_tile_t* x, shard_dtype_t dtype, const void* tile, const double* sums,
                                double count, double eps, int64_t groups, const float* gamma, const float* beta,
                                void* out, void* ws, size_t ws_bytes, hipStream_t stream)
{
    Tile3 t;
    if (!norm_tile(x, dtype, t) || groups < 1 || groups > t.c || t.c % groups != 0) return SHARD_ERR_INVALID;
    if (!(count > 0.0) || !(count < 1e300) || !(eps >= 0.0) || !(eps < 1e300)) return SHARD_ERR_INVALID;
    if (t.n * t.ext[0] * t.ext[1] * t.ext[2] == 0) return SHARD_OK;
    const size_t need = norm_workspace(t, groups);
    if (!tile || !out || !sums || !gamma || !beta || !ws || ws_bytes < need) return SHARD_ERR_INVALID;
    if (!aligned(tile, t.esz) || !aligned(out, t.esz) || !aligned(sums, 8) || !aligned(gamma, 4) ||
        !aligned(beta, 4) || !aligned(ws, 16))
        return SHARD_ERR_INVALID;
    return map_hip(launch_norm_apply(t, dtype, tile, sums, count, eps, groups, gamma, beta, out, ws, stream));
}

}  // extern "C"
