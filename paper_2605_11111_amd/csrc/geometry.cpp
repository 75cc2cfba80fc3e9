// Shard geometry in closed form (host only).
//
// Per axis: output j reads inputs j*S - P + t, t in [0, K), P = (K - 1) / 2;
// the full output has n_out = (G + 2P - K) / S + 1 rows. A shard with interior
// [o, o + L) owns the outputs whose anchor j*S lies in its interior (the
// reading taken of the paper's uneven output chunks, section "ShardTensor"):
//   j0 = ceil(o / S),  j1 = min(ceil((o + L) / S), n_out).
// Its owned outputs read rows [j0*S - P, (j1-1)*S - P + K - 1], so the raw halo
// below / above the interior is
//   r_lo = o - (j0*S - P),   r_hi = (j1-1)*S - P + K - 1 - (o + L - 1),
// the margins are max(0, r) (rows outside the domain are zero padding), and a
// negative r_lo means the first -r_lo interior rows are never read, which the
// convolution skips through pad_lo = min(0, r_lo).
#include <algorithm>

#include "shardconv.h"

namespace {

int64_t cdiv(int64_t a, int64_t b) { return a >= 0 ? (a + b - 1) / b : -((-a) / b); }

}  // namespace

extern "C" shard_status_t shard_conv_geometry(int32_t ndim, const int64_t global_ext[], const int64_t shard_off[],
                                              const int64_t shard_ext[], const int64_t kernel[],
                                              const int64_t stride[], const int64_t sharded_mask[],
                                              int64_t halo_lo[], int64_t halo_hi[], int64_t pad_lo[],
                                              int64_t out_off[], int64_t out_ext[])
{
    if (ndim < 1 || ndim > 3) return SHARD_ERR_INVALID;
    if (!global_ext || !shard_off || !shard_ext || !kernel || !stride || !sharded_mask || !halo_lo ||
        !halo_hi || !pad_lo || !out_off || !out_ext)
        return SHARD_ERR_INVALID;
    const int64_t kLimit = int64_t(1) << 40;
    for (int a = 0; a < ndim; ++a) {
        const int64_t G = global_ext[a], K = kernel[a], S = stride[a], o = shard_off[a], L = shard_ext[a];
        if (G < 1 || G > kLimit || K < 1 || K > kLimit || S < 1 || S > kLimit) return SHARD_ERR_INVALID;
        if (sharded_mask[a]) {
            if (o < 0 || L < 0 || o + L > G) return SHARD_ERR_INVALID;
        } else if (o != 0 || L != G) {
            return SHARD_ERR_INVALID;
        }
    }
    // "same" padding P = (K - 1) / 2 per side needs an odd kernel
    for (int a = 0; a < ndim; ++a)
        if (kernel[a] % 2 == 0) return SHARD_ERR_UNSUPPORTED;
    for (int a = 0; a < ndim; ++a) {
        const int64_t G = global_ext[a], K = kernel[a], S = stride[a], o = shard_off[a], L = shard_ext[a];
        const int64_t P = (K - 1) / 2;
        const int64_t n_out = (G + 2 * P - K) / S + 1;
        if (!sharded_mask[a]) {
            halo_lo[a] = halo_hi[a] = 0;
            pad_lo[a] = P;
            out_off[a] = 0;
            out_ext[a] = n_out;
            continue;
        }
        const int64_t j0 = cdiv(o, S);
        const int64_t j1 = std::min(cdiv(o + L, S), n_out);
        if (j0 >= j1) {
            halo_lo[a] = halo_hi[a] = 0;
            pad_lo[a] = 0;
            out_off[a] = std::min(j0, n_out);
            out_ext[a] = 0;
            continue;
        }
        const int64_t r_lo = o - (j0 * S - P);
        const int64_t r_hi = (j1 - 1) * S - P + K - 1 - (o + L - 1);
        halo_lo[a] = std::max<int64_t>(0, r_lo);
        halo_hi[a] = std::max<int64_t>(0, r_hi);
        pad_lo[a] = std::min<int64_t>(0, r_lo);
        out_off[a] = j0;
        out_ext[a] = j1 - j0;
    }
    return SHARD_OK;
}
