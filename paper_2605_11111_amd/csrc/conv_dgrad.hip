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
// Stride phases. Per axis, tile row p = phi + S*m (phase phi in [0, S)) is
// reached only by taps t = r + S*u with r = (phi + pad) mod S, and then
// jj = m + c - u with c = (phi + pad - r) / S. So each phase is a unit-stride
// forward convolution of dy (zero outside the owned box) with the sub-kernel
// of its taps, flipped and channel-swapped,
//   w_phi[ci][co][u'] = w[co][ci][r + S*(Ku - 1 - u')],   pad' = Ku - 1 - c,
// over the M = ceil((P - phi) / S) rows of that phase, written to every S-th
// tile row through an output map. Unit stride is the single phase phi = 0 with
// the whole flipped kernel and a dense map, which runs on the W-march kernel
// for the 3x3(x3) bf16 shapes. A phase without taps (S > K) is zero-filled.
// SHARDCONV_ALGO=generic takes a direct kernel instead (one thread per tile
// element, over the taps whose phase matches): a structurally different
// cross-check.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {
namespace {

// w_phi[ci][co][u0][u1][u2] = w[co][ci][r0 + S0 (Ku0-1-u0)][r1 + S1 (Ku1-1-u1)][r2 + S2 (Ku2-1-u2)]
struct SubKernel {
    int32_t K[3], Ku[3], r[3], S[3];
};

template <typename T>
__global__ __launch_bounds__(256) void dgrad_weights(const T* __restrict__ w, T* __restrict__ wt, int64_t cin,
                                                     int64_t cout, SubKernel k)
{
    const int64_t taps = int64_t(k.Ku[0]) * k.Ku[1] * k.Ku[2];
    const int64_t total = cin * cout * taps;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        const int64_t u2 = e % k.Ku[2], u1 = (e / k.Ku[2]) % k.Ku[1], u0 = (e / (int64_t(k.Ku[1]) * k.Ku[2])) % k.Ku[0];
        const int64_t co = (e / taps) % cout, ci = e / (taps * cout);
        const int64_t t0 = k.r[0] + int64_t(k.S[0]) * (k.Ku[0] - 1 - u0);
        const int64_t t1 = k.r[1] + int64_t(k.S[1]) * (k.Ku[1] - 1 - u1);
        const int64_t t2 = k.r[2] + int64_t(k.S[2]) * (k.Ku[2] - 1 - u2);
        wt[e] = w[(((co * cin + ci) * k.K[0] + t0) * k.K[1] + t1) * k.K[2] + t2];
    }
}

// zeros at the elements an output map addresses (a phase that no tap reaches)
template <typename T>
__global__ __launch_bounds__(256) void fill_zero_mapped(T* __restrict__ y, int64_t n, int64_t M0, int64_t M1,
                                                        int64_t M2, int64_t c, OutMap om)
{
    const int64_t total = n * M0 * M1 * M2 * c;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        int64_t r = e;
        const int64_t ci = r % c; r /= c;
        const int64_t m2 = r % M2; r /= M2;
        const int64_t m1 = r % M1; r /= M1;
        const int64_t m0 = r % M0;
        const int64_t nn = r / M0;
        y[om.base + nn * om.str[0] + m0 * om.str[1] + m1 * om.str[2] + m2 * om.str[3] + ci] = T(0);
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

// One stride phase of the input gradient as a forward problem on dy.
struct Phase {
    bool empty;     // no tile row has this phase
    bool zero;      // rows of this phase, but no tap reaches them
    SubKernel k;
    Tile3 tf;       // dy as the input tile
    Conv3 cf;       // the unit-stride sub-convolution; cf.O = M
    OutMap om;      // where its rows sit in the tile
};

Phase make_phase(const Tile3& t, const Conv3& cv, const int phi[3])
{
    Phase ph{};
    ph.tf.n = t.n;
    ph.tf.c = cv.cout;
    ph.tf.esz = t.esz;
    ph.cf.cout = t.c;
    int64_t base = 0;
    const int64_t str[3] = {t.P[1] * t.P[2] * t.c, t.P[2] * t.c, t.c};
    for (int a = 0; a < 3; ++a) {
        const int64_t S = cv.S[a], K = cv.K[a];
        const int64_t M = phi[a] < t.P[a] ? ceil_div(t.P[a] - phi[a], S) : 0;
        if (M == 0) ph.empty = true;
        const int64_t r = ((phi[a] + cv.pad[a]) % S + S) % S;
        const int64_t Ku = r < K ? ceil_div(K - r, S) : 0;
        if (Ku == 0) ph.zero = true;
        const int64_t c = (phi[a] + cv.pad[a] - r) / S;  // exact
        ph.k.K[a] = int32_t(K);
        ph.k.Ku[a] = int32_t(std::max<int64_t>(Ku, 1));
        ph.k.r[a] = int32_t(r);
        ph.k.S[a] = int32_t(S);
        ph.tf.P[a] = ph.tf.ext[a] = cv.O[a];
        ph.tf.lo[a] = ph.tf.hi[a] = 0;
        ph.cf.K[a] = ph.k.Ku[a];
        ph.cf.S[a] = 1;
        ph.cf.pad[a] = Ku - 1 - c;
        ph.cf.O[a] = M;
        base += phi[a] * str[a];
        ph.om.str[1 + a] = S * str[a];
    }
    ph.om.base = base;
    ph.om.str[0] = t.P[0] * t.P[1] * t.P[2] * t.c;
    return ph;
}

template <typename F>
void for_each_phase(const Tile3& t, const Conv3& cv, F&& f)
{
    int phi[3];
    for (phi[0] = 0; phi[0] < cv.S[0]; ++phi[0])
        for (phi[1] = 0; phi[1] < cv.S[1]; ++phi[1])
            for (phi[2] = 0; phi[2] < cv.S[2]; ++phi[2]) f(make_phase(t, cv, phi));
}

size_t wt_bytes(const Phase& ph)
{
    return size_t(round_up(ph.cf.cout * ph.tf.c * ph.cf.taps() * ph.tf.esz, 256));
}

// W pairing. A phase whose outputs have 16 channels fills only half of a
// 32-wide matrix tile. With unit stride along W, output row u = 2 u' + p and
// input row u + k - pad = 2 (u' + m) + q for m = floor((p + k - pad) / 2),
// q = (p + k - pad) mod 2, so the phase is also a convolution over the
// W-halved grid with channels (p, ci) out and (q, co) in: dy read as
// [..][O2 / 2][2 cout] and the tile rows as [..][M2 / 2][2 cin] are the same
// bytes (channels-last), and the kernel along W has ceil taps m - mlo,
//   w2[p cin + ci][q cout + co][u0][u1][m'] = w_phi[ci][co][u0][u1][2 (m' + mlo) + q - p + pad]
// (zero where that tap is outside the kernel). 32 output channels fill the
// tile; the zero taps cost (2 ceil(...) ) / K2 - 1 of extra products instead of
// the half tile.
struct Paired {
    bool ok;
    Phase ph;    // the W-halved problem
    int32_t mlo; // first m
};

Paired pair_w(const Tile3& t, const Phase& ph)
{
    Paired pr{};
    pr.ok = false;
    if (force_tiled() || ph.empty || ph.zero || t.c != 16 || ph.k.S[2] != 1 || ph.tf.P[2] % 2 != 0 ||
        ph.cf.O[2] % 2 != 0 || ph.om.str[3] != t.c)
        return pr;
    const int64_t K = ph.cf.K[2], pad = ph.cf.pad[2];
    auto fdiv = [](int64_t a, int64_t b) { return a >= 0 ? a / b : -((-a + b - 1) / b); };
    const int64_t mlo = fdiv(-pad, 2), mhi = fdiv(1 + (K - 1) - pad, 2);
    pr.ph = ph;
    pr.ph.tf.c = 2 * ph.tf.c;
    pr.ph.tf.P[2] = pr.ph.tf.ext[2] = ph.tf.P[2] / 2;
    pr.ph.cf.cout = 2 * ph.cf.cout;
    pr.ph.cf.K[2] = mhi - mlo + 1;
    pr.ph.cf.pad[2] = -mlo;
    pr.ph.cf.O[2] = ph.cf.O[2] / 2;
    pr.ph.om.str[3] = 2 * ph.om.str[3];
    pr.mlo = int32_t(mlo);
    pr.ok = true;
    return pr;
}

template <typename T>
__global__ __launch_bounds__(256) void dgrad_weights_paired(const T* __restrict__ w, T* __restrict__ wt, int64_t cin,
                                                            int64_t cout, SubKernel k, int32_t K2p, int32_t mlo,
                                                            int32_t pad2)
{
    const int64_t taps = int64_t(k.Ku[0]) * k.Ku[1] * K2p;
    const int64_t total = 4 * cin * cout * taps;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
        const int64_t mp = e % K2p, u1 = (e / K2p) % k.Ku[1], u0 = (e / (int64_t(k.Ku[1]) * K2p)) % k.Ku[0];
        const int64_t ic = (e / taps) % (2 * cout), oc = e / (taps * 2 * cout);
        const int64_t p = oc / cin, ci = oc % cin, q = ic / cout, co = ic % cout;
        const int64_t u2 = 2 * (mp + mlo) + q - p + pad2;
        T v = T(0);
        if (u2 >= 0 && u2 < k.Ku[2]) {
            const int64_t t0 = k.r[0] + int64_t(k.S[0]) * (k.Ku[0] - 1 - u0);
            const int64_t t1 = k.r[1] + int64_t(k.S[1]) * (k.Ku[1] - 1 - u1);
            const int64_t t2 = k.r[2] + int64_t(k.S[2]) * (k.Ku[2] - 1 - u2);
            v = w[(((co * cin + ci) * k.K[0] + t0) * k.K[1] + t1) * k.K[2] + t2];
        }
        wt[e] = v;
    }
}

}  // namespace

size_t conv_dgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    if (force_generic()) return 0;
    size_t need = 0;
    for_each_phase(t, cv, [&](const Phase& ph) {
        if (ph.empty || ph.zero) return;
        const Paired pr = pair_w(t, ph);
        const Phase& q = pr.ok ? pr.ph : ph;
        need = std::max(need, wt_bytes(q) + conv_fwd_workspace(q.tf, q.cf, dt));
    });
    return need;
}

hipError_t launch_conv_dgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* dy, const void* w,
                             void* dtile, void* ws, hipStream_t s)
{
    if (!force_generic()) {
        // phases run one after another on the stream and reuse the workspace
        hipError_t err = hipSuccess;
        for_each_phase(t, cv, [&](const Phase& ph) {
            if (err != hipSuccess || ph.empty) return;
            if (ph.zero) {
                const int64_t total = t.n * ph.cf.O[0] * ph.cf.O[1] * ph.cf.O[2] * t.c;
                const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 1 << 16)));
                if (dt == SHARD_BF16)
                    hipLaunchKernelGGL(fill_zero_mapped<bf16_t>, dim3(grid), dim3(256), 0, s,
                                       static_cast<bf16_t*>(dtile), t.n, ph.cf.O[0], ph.cf.O[1], ph.cf.O[2], t.c,
                                       ph.om);
                else
                    hipLaunchKernelGGL(fill_zero_mapped<float>, dim3(grid), dim3(256), 0, s,
                                       static_cast<float*>(dtile), t.n, ph.cf.O[0], ph.cf.O[1], ph.cf.O[2], t.c,
                                       ph.om);
                err = hipGetLastError();
                return;
            }
            char* wt = static_cast<char*>(ws);
            const Paired pr = pair_w(t, ph);
            if (pr.ok) {
                const Phase& q = pr.ph;
                const int64_t total = q.cf.cout * q.tf.c * q.cf.taps();
                const unsigned grid =
                    unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 4096)));
                const int32_t K2p = int32_t(q.cf.K[2]), pad2 = int32_t(ph.cf.pad[2]);
                if (dt == SHARD_BF16)
                    hipLaunchKernelGGL(dgrad_weights_paired<bf16_t>, dim3(grid), dim3(256), 0, s,
                                       static_cast<const bf16_t*>(w), reinterpret_cast<bf16_t*>(wt), t.c, cv.cout,
                                       ph.k, K2p, pr.mlo, pad2);
                else
                    hipLaunchKernelGGL(dgrad_weights_paired<float>, dim3(grid), dim3(256), 0, s,
                                       static_cast<const float*>(w), reinterpret_cast<float*>(wt), t.c, cv.cout,
                                       ph.k, K2p, pr.mlo, pad2);
                err = hipGetLastError();
                if (err == hipSuccess)
                    err = launch_conv_fwd_mapped(q.tf, q.cf, dt, dy, wt, dtile, q.om, wt + wt_bytes(q), s);
                return;
            }
            const int64_t total = t.c * cv.cout * ph.cf.taps();
            const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>(ceil_div(total, 256), 4096)));
            if (dt == SHARD_BF16)
                hipLaunchKernelGGL(dgrad_weights<bf16_t>, dim3(grid), dim3(256), 0, s, static_cast<const bf16_t*>(w),
                                   reinterpret_cast<bf16_t*>(wt), t.c, cv.cout, ph.k);
            else
                hipLaunchKernelGGL(dgrad_weights<float>, dim3(grid), dim3(256), 0, s, static_cast<const float*>(w),
                                   reinterpret_cast<float*>(wt), t.c, cv.cout, ph.k);
            err = hipGetLastError();
            if (err == hipSuccess)
                err = launch_conv_fwd_mapped(ph.tf, ph.cf, dt, dy, wt, dtile, ph.om, wt + wt_bytes(ph), s);
        });
        return err;
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
