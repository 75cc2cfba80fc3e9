// Input gradient of the convolution read back onto the padded tile (the
// backward pass of a shard's convolution: the convolution analogue of
// dL/dx = dL/dz W, ShardTensor section "What Causes High GPU Memory Usage?",
// subsection "An Example of Memory Usage"):
//
//   dtile[n][p][ci] = sum over co, taps t and outputs jj with jj*S + t - pad = p
//                     of w[co][ci][t] * dy[n][jj][co]
//
// for every tile row p, margins included (the margin rows collect the gradient
// that belongs to the neighbours' interiors; shard_halo_pack_margin and
// shard_halo_accumulate return it).
//
// Unit stride: the sum is a forward convolution of dy (zero outside the owned
// output box) with the flipped, channel-transposed kernel
//   w'[ci][co][t'] = w[co][ci][K - 1 - t'],   pad' = K - 1 - pad,
// over the output box P (the padded tile), so it runs on the forward MFMA
// kernels (the W-march kernel for the 3x3(x3) bf16 shapes). Other strides take a
// direct kernel: one thread per tile element, over the taps whose phase matches.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void dgrad_weights(const T* __restrict__ w, T* __restrict__ wt, int64_t cin,
                                                     int64_t cout, int K0, int K1, int K2)
{
    const int64_t taps = int64_t(K0) * K1 * K2;
    const int64_t total = cin * cout * taps;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        // e indexes w'[ci][co][a][b][c]
        const int64_t c = e % K2, b = (e / K2) % K1, a = (e / (int64_t(K1) * K2)) % K0;
        const int64_t co = (e / taps) % cout, ci = e / (taps * cout);
        const int64_t src = (((co * cin + ci) * K0 + (K0 - 1 - a)) * K1 + (K1 - 1 - b)) * K2 + (K2 - 1 - c);
        wt[e] = w[src];
    }
}

struct DgArgs {
    const void* dy;
    const void* w;
    void* dtile;
    int64_t n, cin, cout;
    int64_t P[3], K[3], S[3], pad[3], O[3];
};

template <typename T>
__global__ __launch_bounds__(256) void dgrad_direct(DgArgs a)
{
    const int64_t total = a.n * a.P[0] * a.P[1] * a.P[2] * a.cin;
    const T* dy = static_cast<const T*>(a.dy);
    const T* w = static_cast<const T*>(a.w);
    T* out = static_cast<T*>(a.dtile);
    const int64_t taps = a.K[0] * a.K[1] * a.K[2];
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        int64_t r = e;
        const int64_t ci = r % a.cin; r /= a.cin;
        const int64_t p2 = r % a.P[2]; r /= a.P[2];
        const int64_t p1 = r % a.P[1]; r /= a.P[1];
        const int64_t p0 = r % a.P[0];
        const int64_t nn = r / a.P[0];
        float acc = 0.f;
        for (int64_t k0 = 0; k0 < a.K[0]; ++k0) {
            const int64_t q0 = p0 + a.pad[0] - k0;
            if (q0 < 0 || q0 % a.S[0] != 0 || q0 / a.S[0] >= a.O[0]) continue;
            const int64_t j0 = q0 / a.S[0];
            for (int64_t k1 = 0; k1 < a.K[1]; ++k1) {
                const int64_t q1 = p1 + a.pad[1] - k1;
                if (q1 < 0 || q1 % a.S[1] != 0 || q1 / a.S[1] >= a.O[1]) continue;
                const int64_t j1 = q1 / a.S[1];
                for (int64_t k2 = 0; k2 < a.K[2]; ++k2) {
                    const int64_t q2 = p2 + a.pad[2] - k2;
                    if (q2 < 0 || q2 % a.S[2] != 0 || q2 / a.S[2] >= a.O[2]) continue;
                    const int64_t j2 = q2 / a.S[2];
                    const T* g = dy + (((nn * a.O[0] + j0) * a.O[1] + j1) * a.O[2] + j2) * a.cout;
                    const T* wk = w + ci * taps + (k0 * a.K[1] + k1) * a.K[2] + k2;
                    const int64_t wstride = a.cin * taps;
                    for (int64_t co = 0; co < a.cout; ++co) acc += to_f32(g[co]) * to_f32(wk[co * wstride]);
                }
            }
        }
        out[e] = from_f32<T>(acc);
    }
}

bool unit_stride(const Conv3& cv) { return cv.S[0] == 1 && cv.S[1] == 1 && cv.S[2] == 1; }

// dy as the input tile and the tile's extent as the output box of the
// equivalent forward convolution (unit stride only).
void as_forward(const Tile3& t, const Conv3& cv, Tile3& tf, Conv3& cf)
{
    tf.n = t.n;
    tf.c = cv.cout;
    tf.esz = t.esz;
    cf.cout = t.c;
    for (int k = 0; k < 3; ++k) {
        tf.P[k] = tf.ext[k] = cv.O[k];
        tf.lo[k] = tf.hi[k] = 0;
        cf.K[k] = cv.K[k];
        cf.S[k] = 1;
        cf.pad[k] = cv.K[k] - 1 - cv.pad[k];
        cf.O[k] = t.P[k];
    }
}

size_t wt_bytes(const Tile3& t, const Conv3& cv) { return size_t(round_up(t.c * cv.cout * cv.taps() * t.esz, 256)); }

}  // namespace

size_t conv_dgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    if (!unit_stride(cv) || force_generic()) return 0;
    Tile3 tf;
    Conv3 cf;
    as_forward(t, cv, tf, cf);
    return wt_bytes(t, cv) + conv_fwd_workspace(tf, cf, dt);
}

hipError_t launch_conv_dgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* dy, const void* w,
                             void* dtile, void* ws, hipStream_t s)
{
    if (unit_stride(cv) && !force_generic()) {
        Tile3 tf;
        Conv3 cf;
        as_forward(t, cv, tf, cf);
        char* wt = static_cast<char*>(ws);
        const int64_t total = t.c * cv.cout * cv.taps();
        const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 4096)));
        if (dt == SHARD_BF16)
            hipLaunchKernelGGL(dgrad_weights<bf16_t>, dim3(grid), dim3(256), 0, s, static_cast<const bf16_t*>(w),
                               reinterpret_cast<bf16_t*>(wt), t.c, cv.cout, int(cv.K[0]), int(cv.K[1]), int(cv.K[2]));
        else
            hipLaunchKernelGGL(dgrad_weights<float>, dim3(grid), dim3(256), 0, s, static_cast<const float*>(w),
                               reinterpret_cast<float*>(wt), t.c, cv.cout, int(cv.K[0]), int(cv.K[1]), int(cv.K[2]));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return launch_conv_fwd(tf, cf, dt, dy, wt, dtile, wt + wt_bytes(t, cv), s);
    }
    DgArgs a{};
    a.dy = dy;
    a.w = w;
    a.dtile = dtile;
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
    const int64_t total = t.n * t.P[0] * t.P[1] * t.P[2] * t.c;
    const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 1 << 16)));
    void* args[] = {&a};
    const void* fn = dt == SHARD_BF16 ? reinterpret_cast<const void*>(&dgrad_direct<bf16_t>)
                                      : reinterpret_cast<const void*>(&dgrad_direct<float>);
    return hipLaunchKernel(fn, dim3(grid), dim3(256), args, 0, s);
}

}  // namespace shardconv
