// Direct (untiled) convolution kernels for any shape: one thread per output
// element (forward) or per (weight element, output chunk) (weight gradient).
// They serve shapes outside the tiled MFMA kernels' envelope and give tests a
// second, structurally different GPU implementation to cross-check against.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {
namespace {

struct GenArgs {
    const void* tile;
    const void* w_or_dy;
    void* out;
    float* part;
    int64_t n, cin, cout;
    int64_t P[3], K[3], S[3], pad[3], O[3];
    int64_t chunk, nchunks, ndw;
    int64_t ybase, ys[4];  // forward output map (see OutMap)
    int64_t org[3];        // forward: origin of the computed region (O is its extent)
    Fold fold;             // forward: halo folded into the loads when fold.mask != 0
};

template <typename T>
__global__ __launch_bounds__(256) void fwd_direct(GenArgs a)
{
    const int64_t total = a.n * a.O[0] * a.O[1] * a.O[2] * a.cout;
    const T* tile = static_cast<const T*>(a.tile);
    const T* w = static_cast<const T*>(a.w_or_dy);
    T* y = static_cast<T*>(a.out);
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        int64_t r = e;
        const int64_t co = r % a.cout; r /= a.cout;
        const int64_t o2 = r % a.O[2] + a.org[2]; r /= a.O[2];
        const int64_t o1 = r % a.O[1] + a.org[1]; r /= a.O[1];
        const int64_t o0 = r % a.O[0] + a.org[0];
        const int64_t nn = r / a.O[0];
        float acc = 0.f;
        for (int64_t k0 = 0; k0 < a.K[0]; ++k0) {
            const int64_t i0 = o0 * a.S[0] + k0 - a.pad[0];
            if (i0 < 0 || i0 >= a.P[0]) continue;
            for (int64_t k1 = 0; k1 < a.K[1]; ++k1) {
                const int64_t i1 = o1 * a.S[1] + k1 - a.pad[1];
                if (i1 < 0 || i1 >= a.P[1]) continue;
                for (int64_t k2 = 0; k2 < a.K[2]; ++k2) {
                    const int64_t i2 = o2 * a.S[2] + k2 - a.pad[2];
                    if (i2 < 0 || i2 >= a.P[2]) continue;
                    const T* src = a.fold.mask
                        ? reinterpret_cast<const T*>(fold_voxel(a.fold, static_cast<const char*>(a.tile), nn, i0, i1,
                                                                i2, a.cin * int64_t(sizeof(T))))
                        : tile + (((nn * a.P[0] + i0) * a.P[1] + i1) * a.P[2] + i2) * a.cin;
                    if (!src) continue;
                    const T* wk = w + co * a.cin * a.K[0] * a.K[1] * a.K[2] + (k0 * a.K[1] + k1) * a.K[2] + k2;
                    const int64_t wstride = a.K[0] * a.K[1] * a.K[2];
                    for (int64_t ci = 0; ci < a.cin; ++ci) acc += to_f32(src[ci]) * to_f32(wk[ci * wstride]);
                }
            }
        }
        y[a.ybase + nn * a.ys[0] + o0 * a.ys[1] + o1 * a.ys[2] + o2 * a.ys[3] + co] = from_f32<T>(acc);
    }
}

// part[chunk][tap][co][ci] = sum over the chunk's outputs of dy * x.
template <typename T>
__global__ __launch_bounds__(256) void wgrad_direct(GenArgs a)
{
    const int64_t taps = a.K[0] * a.K[1] * a.K[2];
    const int64_t total = a.ndw * a.nchunks;
    const int64_t nvox = a.n * a.O[0] * a.O[1] * a.O[2];
    const T* tile = static_cast<const T*>(a.tile);
    const T* dy = static_cast<const T*>(a.w_or_dy);
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        const int64_t d = e % a.ndw;
        const int64_t ch = e / a.ndw;
        const int64_t ci = d % a.cin;
        const int64_t co = (d / a.cin) % a.cout;
        const int64_t tap = d / (a.cin * a.cout);
        const int64_t k2 = tap % a.K[2], k1 = (tap / a.K[2]) % a.K[1], k0 = tap / (a.K[2] * a.K[1]);
        float acc = 0.f;
        const int64_t v1 = std::min(nvox, (ch + 1) * a.chunk);
        for (int64_t v = ch * a.chunk; v < v1; ++v) {
            int64_t r = v;
            const int64_t o2 = r % a.O[2]; r /= a.O[2];
            const int64_t o1 = r % a.O[1]; r /= a.O[1];
            const int64_t o0 = r % a.O[0];
            const int64_t nn = r / a.O[0];
            const int64_t i0 = o0 * a.S[0] + k0 - a.pad[0];
            const int64_t i1 = o1 * a.S[1] + k1 - a.pad[1];
            const int64_t i2 = o2 * a.S[2] + k2 - a.pad[2];
            if (i0 < 0 || i0 >= a.P[0] || i1 < 0 || i1 >= a.P[1] || i2 < 0 || i2 >= a.P[2]) continue;
            const T* vox = a.fold.mask
                               ? reinterpret_cast<const T*>(fold_voxel(a.fold, static_cast<const char*>(a.tile), nn,
                                                                       i0, i1, i2, a.cin * int64_t(sizeof(T))))
                               : tile + (((nn * a.P[0] + i0) * a.P[1] + i1) * a.P[2] + i2) * a.cin;
            if (!vox) continue;
            const float xv = to_f32(vox[ci]);
            acc += to_f32(dy[v * a.cout + co]) * xv;
        }
        a.part[e] = acc;
    }
}

// dw[co][ci][tap] = sum over chunks, in chunk order, of part[chunk][tap][co][ci].
__global__ __launch_bounds__(256) void wgrad_direct_reduce(GenArgs a)
{
    const int64_t taps = a.K[0] * a.K[1] * a.K[2];
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < a.ndw; e += int64_t(gridDim.x) * 256) {
        const int64_t tap = e % taps;
        const int64_t ci = (e / taps) % a.cin;
        const int64_t co = e / (taps * a.cin);
        const int64_t d = (tap * a.cout + co) * a.cin + ci;
        float acc = 0.f;
        for (int64_t ch = 0; ch < a.nchunks; ++ch) acc += a.part[ch * a.ndw + d];
        static_cast<float*>(a.out)[e] = acc;
    }
}

GenArgs make_args(const Tile3& t, const Conv3& cv)
{
    GenArgs a{};
    a.n = t.n;
    a.cin = t.c;
    a.cout = cv.cout;
    for (int k = 0; k < 3; ++k) {
        a.P[k] = t.P[k];
        a.K[k] = cv.K[k];
        a.S[k] = cv.S[k];
        a.pad[k] = cv.pad[k];
        a.O[k] = cv.O[k];
    }
    a.ndw = cv.cout * t.c * cv.taps();
    const int64_t nvox = t.n * cv.out_voxels();
    a.chunk = std::max<int64_t>(256, ceil_div(nvox, 256));
    a.nchunks = std::max<int64_t>(1, ceil_div(nvox, a.chunk));
    return a;
}

unsigned grid_for(int64_t total) { return unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 1 << 16))); }

}  // namespace

size_t generic_wgrad_workspace(const Tile3& t, const Conv3& cv)
{
    GenArgs a = make_args(t, cv);
    return size_t(a.nchunks * a.ndw) * sizeof(float);
}

hipError_t generic_conv_fwd(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* w,
                            void* y, const OutMap& om, const Region& rg, const Fold* fold, hipStream_t s)
{
    GenArgs a = make_args(t, cv);
    for (int k = 0; k < 3; ++k) {
        a.O[k] = rg.ext[k];
        a.org[k] = rg.org[k];
    }
    if (fold) a.fold = *fold;
    a.ybase = om.base;
    for (int k = 0; k < 4; ++k) a.ys[k] = om.str[k];
    a.tile = tile;
    a.w_or_dy = w;
    a.out = y;
    void* args[] = {&a};
    const int64_t total = t.n * rg.ext[0] * rg.ext[1] * rg.ext[2] * cv.cout;
    if (total == 0) return hipSuccess;
    const void* fn = dt == SHARD_BF16 ? reinterpret_cast<const void*>(&fwd_direct<bf16_t>)
                                      : reinterpret_cast<const void*>(&fwd_direct<float>);
    return hipLaunchKernel(fn, dim3(grid_for(total)), dim3(256), args, 0, s);
}

hipError_t generic_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                              float* dw, void* ws, const Fold* fold, hipStream_t s)
{
    GenArgs a = make_args(t, cv);
    if (fold) a.fold = *fold;
    a.tile = tile;
    a.w_or_dy = dy;
    a.out = dw;
    a.part = static_cast<float*>(ws);
    void* args[] = {&a};
    const void* fn = dt == SHARD_BF16 ? reinterpret_cast<const void*>(&wgrad_direct<bf16_t>)
                                      : reinterpret_cast<const void*>(&wgrad_direct<float>);
    hipError_t e = hipLaunchKernel(fn, dim3(grid_for(a.ndw * a.nchunks)), dim3(256), args, 0, s);
    if (e != hipSuccess) return e;
    return hipLaunchKernel(reinterpret_cast<const void*>(&wgrad_direct_reduce), dim3(grid_for(a.ndw)), dim3(256),
                           args, 0, s);
}

}  // namespace shardconv
