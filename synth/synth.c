/*
 * Seeded synthetic tensors for the shard halo-convolution workloads.
 *
 * This module only draws input values. It holds none of the halo or
 * convolution arithmetic, and both the CPU oracle and the GPU path take their
 * inputs from it, so the two sides always see bit-identical operands.
 *
 * Every element of a logical full-domain tensor [N][C][X0][X1][X2] (missing
 * spatial axes have extent 1) is a pure function of (seed, stream, logical
 * linear index), so any sub-box can be produced on its own and equals the
 * same slice of the full tensor bit for bit.
 *
 * Counter-based hash: the SplitMix64 output function (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014; the mix64
 * finaliser of java.util.SplittableRandom) applied to the state
 * (key << 40) + counter, where key = (seed << 4) | stream.
 *
 * Distributions, all computed in binary64 and then rounded once to the output
 * type (binary32 round-to-nearest-even, then bfloat16 round-to-nearest-even):
 *   UNIFORM(a, b)        a + (b - a) * u,  u = top 53 bits / 2^53
 *   NORMAL(mean, std)    Box-Muller cosine branch on counters 2i and 2i+1
 *   SMOOTH(std, sigma)   white NORMAL(0,1) noise, periodic in every spatial axis
 *                        of the full domain, filtered separably with a Gaussian
 *                        of width sigma truncated at R = floor(4 sigma + 0.5),
 *                        weights normalised to sum 1, then scaled to unit
 *                        marginal variance and multiplied by std
 *   INT(lo, hi)          integer lo + floor(u * (hi - lo + 1))
 *   SPARSE_INT(lo, hi, p) INT(lo, hi) with probability p (decided by a second
 *                        counter stream), otherwise 0
 * Positions of the requested box that lie outside the full domain along a
 * spatial axis are written as 0.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared synth.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

enum { SYNTH_UNIFORM = 0, SYNTH_NORMAL = 1, SYNTH_SMOOTH = 2, SYNTH_INT = 3, SYNTH_SPARSE_INT = 4 };
enum { SYNTH_OUT_F64 = 0, SYNTH_OUT_F32 = 1, SYNTH_OUT_BF16 = 2 };

typedef struct {
    uint64_t seed;
    int32_t stream;
    int32_t dist;
    double p0, p1, p2;
    int32_t ndim;     /* number of real spatial axes (1..3); they are the last ndim of X0..X2 */
    int32_t pad_;
    int64_t full[5];  /* N, C, X0, X1, X2 */
} synth_spec_t;

static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

static inline uint64_t hash_at(uint64_t key, uint64_t ctr)
{
    return mix64((key << 40) + ctr + 0x9e3779b97f4a7c15ULL);
}

static inline double unit53(uint64_t h) { return (double)(h >> 11) * 0x1.0p-53; }

static inline double normal_at(uint64_t key, uint64_t idx)
{
    double u1 = 1.0 - unit53(hash_at(key, 2 * idx));     /* (0, 1] */
    double u2 = unit53(hash_at(key, 2 * idx + 1));       /* [0, 1) */
    return sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
}

static inline uint16_t f32_to_bf16_rne(float f)
{
    uint32_t b;
    memcpy(&b, &f, 4);
    if ((b & 0x7f800000u) == 0x7f800000u) return (uint16_t)((b >> 16) | ((b & 0xffffu) ? 0x40u : 0u));
    b += 0x7fffu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

static inline void store(void* out, int out_type, int64_t pos, double v)
{
    if (out_type == SYNTH_OUT_F64) {
        ((double*)out)[pos] = v;
    } else if (out_type == SYNTH_OUT_F32) {
        ((float*)out)[pos] = (float)v;
    } else {
        ((uint16_t*)out)[pos] = f32_to_bf16_rne((float)v);
    }
}

static inline int64_t wrap(int64_t i, int64_t g)
{
    int64_t r = i % g;
    return r < 0 ? r + g : r;
}

static double point_value(const synth_spec_t* s, uint64_t key, uint64_t idx)
{
    switch (s->dist) {
    case SYNTH_UNIFORM:
        return s->p0 + (s->p1 - s->p0) * unit53(hash_at(key, idx));
    case SYNTH_NORMAL:
        return s->p0 + s->p1 * normal_at(key, idx);
    case SYNTH_INT: {
        double span = s->p1 - s->p0 + 1.0;
        return s->p0 + floor(unit53(hash_at(key, idx)) * span);
    }
    case SYNTH_SPARSE_INT: {
        double span = s->p1 - s->p0 + 1.0;
        double keep = unit53(hash_at(key ^ 0x5ULL, idx));
        if (keep >= s->p2) return 0.0;
        return s->p0 + floor(unit53(hash_at(key, idx)) * span);
    }
    default:
        return 0.0;
    }
}

/* Gaussian filtered, periodic, unit-variance smooth field for one (n, c) channel
 * over the clipped spatial box [a, b). Writes scaled values to out at the given
 * channels-last positions. */
static int smooth_channel(const synth_spec_t* s, uint64_t key, int64_t n, int64_t c,
                          const int64_t a[3], const int64_t b[3], const int64_t blo[3],
                          const int64_t bext[3], int64_t bc, int64_t n_out, int64_t c_out,
                          int out_type, void* out)
{
    const int64_t* G = s->full + 2;
    const double sigma = s->p2;
    const int R = (int)floor(4.0 * sigma + 0.5);
    int Rk[3];
    for (int k = 0; k < 3; ++k) Rk[k] = (k >= 3 - s->ndim) ? R : 0;

    double* g = (double*)malloc(sizeof(double) * (size_t)(2 * R + 1));
    if (!g) return 1;
    double gsum = 0.0;
    for (int t = -R; t <= R; ++t) {
        g[t + R] = exp(-(double)t * (double)t / (2.0 * sigma * sigma));
        gsum += g[t + R];
    }
    double g2 = 0.0;
    for (int t = 0; t <= 2 * R; ++t) {
        g[t] /= gsum;
        g2 += g[t] * g[t];
    }
    const double scale = s->p1 / pow(sqrt(g2), (double)s->ndim);
    /* per-axis weights: the Gaussian on filtered axes, the identity on the others */
    static const double one = 1.0;
    const double* gk[3];
    for (int k = 0; k < 3; ++k) gk[k] = Rk[k] ? g : &one;

    const int64_t e0 = b[0] - a[0], e1 = b[1] - a[1], e2 = b[2] - a[2];
    const int64_t p0 = e0 + 2 * Rk[0], p1 = e1 + 2 * Rk[1];
    double* P1 = (double*)malloc(sizeof(double) * (size_t)(p0 * p1 * e2));
    double* P2 = (double*)malloc(sizeof(double) * (size_t)(p0 * e1 * e2));
    if (!P1 || !P2) {
        free(g); free(P1); free(P2);
        return 1;
    }
    const uint64_t chan_base = ((uint64_t)n * (uint64_t)s->full[1] + (uint64_t)c);

    /* pass 1: along X2, noise generated on the fly (periodic wrap) */
#pragma omp parallel
    {
        double* row = (double*)malloc(sizeof(double) * (size_t)(e2 + 2 * Rk[2]));
#pragma omp for collapse(2) schedule(static)
        for (int64_t i = 0; i < p0; ++i) {
            for (int64_t j = 0; j < p1; ++j) {
                int64_t x0 = wrap(a[0] - Rk[0] + i, G[0]);
                int64_t x1 = wrap(a[1] - Rk[1] + j, G[1]);
                uint64_t base = ((chan_base * (uint64_t)G[0] + (uint64_t)x0) * (uint64_t)G[1] + (uint64_t)x1) * (uint64_t)G[2];
                for (int64_t m = 0; m < e2 + 2 * Rk[2]; ++m) {
                    int64_t x2 = wrap(a[2] - Rk[2] + m, G[2]);
                    row[m] = normal_at(key, base + (uint64_t)x2);
                }
                double* dst = P1 + (i * p1 + j) * e2;
                for (int64_t m = 0; m < e2; ++m) {
                    double acc = 0.0;
                    for (int t = 0; t <= 2 * Rk[2]; ++t) acc += gk[2][t] * row[m + t];
                    dst[m] = acc;
                }
            }
        }
        free(row);
    }
    /* pass 2: along X1 */
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < p0; ++i) {
        for (int64_t j = 0; j < e1; ++j) {
            double* dst = P2 + (i * e1 + j) * e2;
            for (int64_t m = 0; m < e2; ++m) {
                double acc = 0.0;
                for (int t = 0; t <= 2 * Rk[1]; ++t)
                    acc += gk[1][t] * P1[(i * p1 + j + t) * e2 + m];
                dst[m] = acc;
            }
        }
    }
    /* pass 3: along X0, scale, round and scatter into the channels-last box */
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < e0; ++i) {
        for (int64_t j = 0; j < e1; ++j) {
            for (int64_t m = 0; m < e2; ++m) {
                double acc = 0.0;
                for (int t = 0; t <= 2 * Rk[0]; ++t)
                    acc += gk[0][t] * P2[((i + t) * e1 + j) * e2 + m];
                int64_t q0 = a[0] + i - blo[0], q1 = a[1] + j - blo[1], q2 = a[2] + m - blo[2];
                int64_t pos = (((n_out * bext[0] + q0) * bext[1] + q1) * bext[2] + q2) * bc + c_out;
                store(out, out_type, pos, scale * acc);
            }
        }
    }
    free(g);
    free(P1);
    free(P2);
    return 0;
}

/* Fill the box [lo, hi) of the logical [N][C][X0][X1][X2] tensor into a dense
 * channels-last buffer [n][x0][x1][x2][c] of extents (hi - lo).
 * Returns 0 on success, 1 on a bad argument or an allocation failure. */
int synth_fill(const synth_spec_t* s, const int64_t lo[5], const int64_t hi[5], int out_type, void* out)
{
    if (!s || !lo || !hi || !out || s->ndim < 1 || s->ndim > 3) return 1;
    for (int k = 0; k < 5; ++k) {
        if (hi[k] < lo[k] || s->full[k] < 1) return 1;
    }
    if (lo[0] < 0 || hi[0] > s->full[0] || lo[1] < 0 || hi[1] > s->full[1]) return 1;
    if (out_type < 0 || out_type > 2) return 1;
    const uint64_t key = (s->seed << 4) | ((uint64_t)s->stream & 0xfu);
    const int64_t bn = hi[0] - lo[0], bc = hi[1] - lo[1];
    const int64_t bext[3] = {hi[2] - lo[2], hi[3] - lo[3], hi[4] - lo[4]};
    const int64_t blo[3] = {lo[2], lo[3], lo[4]};
    const int64_t total = bn * bc * bext[0] * bext[1] * bext[2];
    if (total == 0) return 0;

    /* zero everything first: positions outside the domain stay 0 */
    size_t esz = out_type == SYNTH_OUT_F64 ? 8 : (out_type == SYNTH_OUT_F32 ? 4 : 2);
    memset(out, 0, (size_t)total * esz);

    int64_t a[3], b[3];
    for (int k = 0; k < 3; ++k) {
        a[k] = blo[k] < 0 ? 0 : blo[k];
        int64_t g = s->full[2 + k];
        b[k] = hi[2 + k] > g ? g : hi[2 + k];
        if (b[k] <= a[k]) return 0;
    }

    if (s->dist == SYNTH_SMOOTH) {
        if (!(s->p2 > 0.0)) return 1;
        for (int64_t n = lo[0]; n < hi[0]; ++n)
            for (int64_t c = lo[1]; c < hi[1]; ++c)
                if (smooth_channel(s, key, n, c, a, b, blo, bext, bc, n - lo[0], c - lo[1], out_type, out))
                    return 1;
        return 0;
    }
    if (s->dist < 0 || s->dist > SYNTH_SPARSE_INT) return 1;

    const int64_t* F = s->full;
    const int64_t e0 = b[0] - a[0], e1 = b[1] - a[1], e2 = b[2] - a[2];
#pragma omp parallel for collapse(3) schedule(static)
    for (int64_t n = lo[0]; n < hi[0]; ++n) {
        for (int64_t i = 0; i < e0; ++i) {
            for (int64_t j = 0; j < e1; ++j) {
                int64_t x0 = a[0] + i, x1 = a[1] + j;
                for (int64_t m = 0; m < e2; ++m) {
                    int64_t x2 = a[2] + m;
                    int64_t q0 = x0 - blo[0], q1 = x1 - blo[1], q2 = x2 - blo[2];
                    int64_t pos0 = ((((n - lo[0]) * bext[0] + q0) * bext[1] + q1) * bext[2] + q2) * bc;
                    for (int64_t c = lo[1]; c < hi[1]; ++c) {
                        uint64_t idx = ((((uint64_t)n * (uint64_t)F[1] + (uint64_t)c) * (uint64_t)F[2] + (uint64_t)x0) *
                                            (uint64_t)F[3] + (uint64_t)x1) * (uint64_t)F[4] + (uint64_t)x2;
                        store(out, out_type, pos0 + (c - lo[1]), point_value(s, key, idx));
                    }
                }
            }
        }
    }
    return 0;
}

/* binary32 -> bfloat16 round-to-nearest-even, exposed so its tie handling can be tested */
void synth_round_bf16(const float* in, uint16_t* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne(in[i]);
}

int synth_threads(void) { return omp_get_max_threads(); }
