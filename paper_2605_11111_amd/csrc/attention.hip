// One block step of ring attention (the paper's first benchmark, section
// "Performance Benchmarks", subsection "Ring Attention"): the local queries
// attend to the key/value block the device holds, and the result is merged in
// log space into the running (output, log-normaliser) state.
//
// Flash-style forward on v_mfma_f32_32x32x16_bf16, per (batch*head, 256-query
// tile) workgroup of four waves, each wave owning 64 queries as two 32-query
// tiles:
//  * Scores are computed transposed, S^T = K Q^T (M = 32 keys, N = 32 queries,
//    K = head dim): the accumulator lane (g, n) then holds 16 keys of query n,
//    so the softmax statistics of a query live in one lane pair (g = 0, 1),
//    joined by one v_permlane32_swap. The Q^T fragments (B operand) stay in
//    registers for the whole key loop.
//  * O^T = V^T P^T (M = 32 head-dim rows, N = 32 queries, K = 32 keys in two
//    steps). The B operand P^T is the exponentiated score accumulator itself,
//    rounded to bf16, with no data movement: the MFMA's K slots of lane half g
//    are mapped to the keys that lane holds (keys 16c + 4g + 0..3 and
//    16c + 8 + 4g + 0..3 for step c), and the A operand V^T is read in the same
//    key order with ds_read_b64_tr_b16 (transpose on read). A query's rescale
//    factor is then one scalar per lane.
//  * K and V blocks of 32 keys are staged by direct global->LDS loads, double
//    buffered, 16-byte units XOR-swizzled by key so that the fragment reads are
//    free of bank conflicts; keys past the block end load as zero and are
//    masked to -inf in the scores, queries past the end load as zero and are
//    not stored.
//  * Softmax runs in base 2 on fp32 (scores scaled by scale * log2 e) against a
//    reference max that moves only when a block's scores exceed it by more than
//    2^8 (the rescale of O and l is then a rare wave-uniform branch); the
//    log-normaliser is m + log2(l), converted to natural log for the state. The
//    merge with the stored state happens in the epilogue.
#include <algorithm>
#include <type_traits>

#include "attention.h"
#include "common.h"

namespace shardconv {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_a;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_a;
typedef __attribute__((ext_vector_type(16))) float f32x16_a;

#define SC_LDSA(p) ((__attribute__((address_space(3))) void*)(p))

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSlack = 8.f;  // log2 headroom of the lazily updated reference max

struct AttnArgs {
    const char* q;
    const char* k;
    const char* v;
    float* o;
    float* lse;
    int32_t sq, sk;
    int32_t nqt;       // 256-query tiles per (batch, head)
    uint32_t nblocks;  // batch * heads * nqt
    float c2;          // scale * log2 e
    int32_t first;
};

template <int D>
struct AttnCfg {
    static constexpr int QT = 2;               // 32-query tiles per wave
    static constexpr int QB = 4 * 32 * QT;     // queries per workgroup
    static constexpr int KB = 32;              // keys per block
    static constexpr int NC = D / 16;          // MFMA K steps over the head dim
    static constexpr int NDT = D / 32;         // 32-row head-dim tiles of O^T
    static constexpr int ROWB = D * 2;         // bytes per key row
    static constexpr int UPR = ROWB / 16;      // 16-byte units per row
    static constexpr int KV_BYTES = KB * ROWB; // one K or V block
    static constexpr int NLD = KV_BYTES / 4096;  // direct loads per matrix per block (256 lanes x 16 B)
    static constexpr int STAGE = 2 * KV_BYTES;   // K block, then V block
    static constexpr int LDS = 2 * STAGE;        // double buffered
    static_assert(D == 64 || D == 128, "head dim 64 or 128");
    static_assert(KV_BYTES % 4096 == 0, "whole direct loads");
};

// swizzled 16-byte slot of unit u of key row `key`
template <int D>
__device__ __forceinline__ constexpr int k_slot(int key, int u)
{
    return u ^ (key & (AttnCfg<D>::UPR - 1));
}
__device__ __forceinline__ constexpr int v_slot(int key, int u) { return u ^ (2 * (key & 3)); }

// f(integral_constant<int, i>) for i = 0 .. N - 1 (compile-time indices)
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f)
{
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}

template <int D>
__global__ __launch_bounds__(256, 1) void attn_block(AttnArgs a)
{
    using C = AttnCfg<D>;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    const uint32_t L = uint32_t(xcd_remap(blockIdx.x, gridDim.x));
    const uint32_t bh = L / uint32_t(a.nqt), qt = L - bh * uint32_t(a.nqt);
    const int q0 = int(qt) * C::QB + wave * 32 * C::QT;

    // Q^T fragments (B operand of S^T): lane (g, n) holds q[n][16c + 8g .. + 8]
    uint4 qf[C::QT][C::NC];
    {
        const uint4* qm = reinterpret_cast<const uint4*>(a.q + int64_t(bh) * a.sq * C::ROWB);
#pragma unroll
        for (int t = 0; t < C::QT; ++t) {
            const int qi = q0 + 32 * t + ln;
#pragma unroll
            for (int c = 0; c < C::NC; ++c)
                qf[t][c] = qi < a.sq ? qm[int64_t(qi) * C::UPR + 2 * c + g] : make_uint4(0, 0, 0, 0);
        }
    }

    // staging: load i of thread tid fills LDS bytes i*4096 + tid*16 of a block,
    // i.e. key row r, slot s; it reads unit k_slot/v_slot^-1 of that key. Step kb
    // stages K of block kb + 1 and V of block kb (V runs one block behind: step kb
    // multiplies the probabilities of block kb - 1); blocks past the end load as
    // zero, so every step issues the same loads.
    const int64_t kv_bytes = int64_t(a.sk) * C::ROWB;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.k) + int64_t(bh) * kv_bytes, short(0), int(uint32_t(kv_bytes)), 0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.v) + int64_t(bh) * kv_bytes, short(0), int(uint32_t(kv_bytes)), 0x00020000);
    auto stage = [&](int kbk, int kbv, int buf) {
        char* dst = lds + buf * C::STAGE + wave * 1024;
#pragma unroll
        for (int i = 0; i < C::NLD; ++i) {
            const int byte = i * 4096 + tid * 16;
            const int r = byte / C::ROWB, sl = (byte % C::ROWB) / 16;
            const int kk = kbk * C::KB + r, kv = kbv * C::KB + r;
            const uint32_t ku = uint32_t(kk) * C::ROWB + uint32_t(k_slot<D>(r, sl)) * 16;
            const uint32_t vu = uint32_t(kv) * C::ROWB + uint32_t(v_slot(r, sl)) * 16;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, SC_LDSA(dst + i * 4096), 16,
                                                     kbk >= 0 && kk < a.sk ? ku : 0xFFFFFFC0u, 0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, SC_LDSA(dst + C::KV_BYTES + i * 4096), 16,
                                                     kbv >= 0 && kv < a.sk ? vu : 0xFFFFFFC0u, 0, 0, 0);
        }
    };

    f32x16_a o[C::QT][C::NDT];
    float m[C::QT], l[C::QT];
#pragma unroll
    for (int t = 0; t < C::QT; ++t) {
        m[t] = -__builtin_inff();
        l[t] = 0.f;
#pragma unroll
        for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[t][dt][r] = 0.f;
    }

    // fragment read addresses (bytes within a staged block). K: lane (g, key n)
    // reads unit 2c + g of its key, slot (2c + g) ^ (n % UPR) = 2 (c ^ zh) + (g ^ zl)
    // with zh = (n % UPR) / 2, zl = n % 2.
    const uint32_t lds0 = lds_addr(lds);
    const int zk = ln & (C::UPR - 1);
    const uint32_t kl = uint32_t(ln * C::ROWB + 16 * (g ^ (zk & 1)));
    const uint32_t kzh = uint32_t(zk >> 1);
    // V^T: within a 16-lane group G, lane i addresses key row 16c + 8h + 4(G/2) + i/4
    // at head-dim columns 32dt + 16(G%2) + 4(i%4): unit 4dt + x (x < 4), slot
    // (4dt + x) ^ 2(i/4) = 4 (dt ^ yb) + (x ^ 2 y1) with yb = i/8, y1 = (i/4) % 2.
    // The dt part is an immediate offset; yb moves even dt by +64 B, odd dt by -64.
    const int G = lane >> 4, ii = lane & 15;
    const int vx = 2 * (G & 1) + ((ii & 3) >> 1), vy1 = (ii >> 2) & 1, vyb = ii >> 3;
    const uint32_t vcom = uint32_t((4 * (G >> 1) + (ii >> 2)) * C::ROWB + 16 * (vx ^ (2 * vy1)) + 8 * (ii & 1));
    const uint32_t vbe = vcom + 64u * uint32_t(vyb), vbo = vcom - 64u * uint32_t(vyb);
    const int nkb = (a.sk + C::KB - 1) / C::KB;
    // Step kb (software pipelined over key blocks): the score MFMAs of block kb,
    // then the O^T MFMAs of block kb - 1 with the masking, row max and
    // exponentials of block kb between them - a wave issues in order, so VALU
    // work has to sit between MFMAs to run in their shadow (sched_group_barrier
    // lays the streams out so). The probabilities alternate between two register
    // sets (pA, pB). When block kb moves the reference max, l is rescaled at once
    // and O at the start of step kb + 1, after the O^T MFMAs of block kb - 1.
    f32x16_a sc[C::QT];
    uint32_t pA[C::QT][2][4], pB[C::QT][2][4];
    float alpha[C::QT];
    bool resc = false;
    auto step = [&](int kb, uint32_t (&pn)[C::QT][2][4], const uint32_t (&pp)[C::QT][2][4], auto do_s_c,
                    auto do_pv_c) {
        constexpr bool DO_S = decltype(do_s_c)::value, DO_PV = decltype(do_pv_c)::value;
        const int buf = kb & 1;
        stage(kb + 1 < nkb ? kb + 1 : -1, kb < nkb ? kb : -1, buf ^ 1);
        wait_vm_barrier<2 * C::NLD>();
        const uint32_t base = lds0 + uint32_t(buf * C::STAGE);
        uint2 vr[2][2][C::NDT];
        const uint32_t ve = base + vbe, vo = base + vbo;
        auto vread = [&](auto c_c, auto h_c, auto dt_c) {
            constexpr int c = decltype(c_c)::value, h = decltype(h_c)::value, dt = decltype(dt_c)::value;
            constexpr int off = C::KV_BYTES + (16 * c + 8 * h) * C::ROWB + 64 * dt;
            return lds_read_tr16_b64<off>((dt & 1) ? vo : ve);
        };
        auto vreads = [&](auto c_c) {
            constexpr int c = decltype(c_c)::value;
            static_for<2>([&](auto h_c) {
                static_for<C::NDT>([&](auto dt_c) {
                    vr[c][decltype(h_c)::value][decltype(dt_c)::value] = vread(c_c, h_c, dt_c);
                });
            });
        };
        if (DO_PV) {
            vreads(std::integral_constant<int, 0>{});
            if (resc) {
#pragma unroll
                for (int t = 0; t < C::QT; ++t)
#pragma unroll
                    for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
                        for (int r = 0; r < 16; ++r) o[t][dt][r] *= alpha[t];
            }
        }
        if (DO_S) {
#pragma unroll
            for (int t = 0; t < C::QT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) sc[t][r] = 0.f;
            const uint32_t kb0 = base + kl;
            auto kaddr = [&](int c) { return kb0 + 32u * (uint32_t(c) ^ kzh); };
            lds_u32x4 kf[2];
            kf[0] = lds_read_b128(kaddr(0));
#pragma unroll
            for (int c = 0; c < C::NC; ++c) {
                if (c + 1 < C::NC) {
                    kf[(c + 1) & 1] = lds_read_b128(kaddr(c + 1));
                    lds_wait<1>();
                } else {
                    lds_wait<0>();
                }
                lds_ready(kf[c & 1]);
#pragma unroll
                for (int t = 0; t < C::QT; ++t)
                    sc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_a, kf[c & 1]),
                                                                    __builtin_bit_cast(bf16x8_a, qf[t][c]), sc[t], 0,
                                                                    0, 0);
            }
        }
        if (DO_PV) {
            lds_wait<0>();
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int dt = 0; dt < C::NDT; ++dt) lds_ready(vr[0][h][dt]);
            vreads(std::integral_constant<int, 1>{});
        }
        auto pv = [&](int c) {
#pragma unroll
            for (int dt = 0; dt < C::NDT; ++dt) {
                const uint4 af = make_uint4(vr[c][0][dt].x, vr[c][0][dt].y, vr[c][1][dt].x, vr[c][1][dt].y);
#pragma unroll
                for (int t = 0; t < C::QT; ++t) {
                    const uint4 bf = make_uint4(pp[t][c][0], pp[t][c][1], pp[t][c][2], pp[t][c][3]);
                    o[t][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_a, af),
                                                                       __builtin_bit_cast(bf16x8_a, bf), o[t][dt],
                                                                       0, 0, 0);
                }
            }
        };
        // O^T MFMAs of block kb - 1, first half | mask and row max of block kb
        if (DO_PV) pv(0);
        float mx[C::QT];
        if (DO_S) {
            const int kleft = a.sk - kb * C::KB;
            if (kleft < C::KB) {
#pragma unroll
                for (int t = 0; t < C::QT; ++t)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (8 * (r >> 2) + 4 * g + (r & 3) >= kleft) sc[t][r] = -__builtin_inff();
            }
            bool need = false;
#pragma unroll
            for (int t = 0; t < C::QT; ++t) {
                float v = sc[t][0];
#pragma unroll
                for (int r = 1; r < 16; ++r) v = fmaxf(v, sc[t][r]);
                const uint32_t u = __float_as_uint(v);
                const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
                mx[t] = fmaxf(v, __uint_as_float(g ? p[0] : p[1])) * a.c2;
                need |= mx[t] > m[t] + kSlack;
            }
            // the reference max moves for every lane when any lane needs it to
            resc = __builtin_amdgcn_ballot_w64(need) != 0;
#pragma unroll
            for (int t = 0; t < C::QT; ++t) {
                const float mn = resc ? fmaxf(m[t], mx[t]) : m[t];
                alpha[t] = __builtin_amdgcn_exp2f(m[t] - mn);
                m[t] = mn;
            }
        }
        if (DO_PV && DO_S) {
#pragma unroll
            for (int i = 0; i < C::NDT * C::QT; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
            }
        }
        if (DO_PV) {
            lds_wait<0>();
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int dt = 0; dt < C::NDT; ++dt) lds_ready(vr[1][h][dt]);
        }
        // O^T MFMAs of block kb - 1, second half | exponentials of block kb
        if (DO_PV) pv(1);
        if (DO_S) {
#pragma unroll
            for (int t = 0; t < C::QT; ++t) {
                float x[16];
                float sum = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    x[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[t][r], a.c2, -m[t]));
                    sum += x[r];
                }
                const uint32_t u = __float_as_uint(sum);
                const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
                l[t] = l[t] * alpha[t] + sum + __uint_as_float(g ? p[0] : p[1]);
#pragma unroll
                for (int c = 0; c < 2; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const bf16x2_a pk = {__bf16(x[8 * c + 2 * e]), __bf16(x[8 * c + 2 * e + 1])};
                        pn[t][c][e] = __builtin_bit_cast(uint32_t, pk);
                    }
            }
        }
        if (DO_PV && DO_S) {
#pragma unroll
            for (int i = 0; i < C::NDT * C::QT; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
            }
        }
        // every wave is done with this buffer before the next step refills it
        __syncthreads();
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    stage(0, -1, 0);
    step(0, pA, pB, T_{}, F_{});
    int kb = 1;
    for (; kb + 1 < nkb; kb += 2) {
        step(kb, pB, pA, T_{}, T_{});
        step(kb + 1, pA, pB, T_{}, T_{});
    }
    if (kb < nkb) {
        step(kb, pB, pA, T_{}, T_{});
        step(kb + 1, pA, pB, F_{}, T_{});
    } else {
        step(kb, pB, pA, F_{}, T_{});
    }

    // epilogue: lane (g, n) holds head-dim rows 32dt + 8j + 4g + e (e < 4) of
    // query q0 + 32t + n; merge with the stored state
    const int64_t orow = int64_t(bh) * a.sq;
#pragma unroll
    for (int t = 0; t < C::QT; ++t) {
        const int qi = q0 + 32 * t + ln;
        if (qi >= a.sq) continue;
        const float lse_b = (m[t] + __builtin_amdgcn_logf(l[t])) * kLn2;
        const float inv = 1.f / l[t];
        float wa = 0.f, wb = inv, lse_n = lse_b;
        if (!a.first) {
            const float old = a.lse[orow + qi];
            const float hi = fmaxf(old, lse_b);
            const float ea = __builtin_amdgcn_exp2f((old - hi) * kLog2e);
            const float eb = __builtin_amdgcn_exp2f((lse_b - hi) * kLog2e);
            const float tot = ea + eb;
            lse_n = hi + __builtin_amdgcn_logf(tot) * kLn2;
            wa = ea / tot;
            wb = eb / tot * inv;
        }
        float4* orow_p = reinterpret_cast<float4*>(a.o + (orow + qi) * D);
#pragma unroll
        for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d4 = (32 * dt + 8 * j + 4 * g) / 4;
                float4 r;
                r.x = o[t][dt][4 * j + 0] * wb;
                r.y = o[t][dt][4 * j + 1] * wb;
                r.z = o[t][dt][4 * j + 2] * wb;
                r.w = o[t][dt][4 * j + 3] * wb;
                if (!a.first) {
                    const float4 ov = orow_p[d4];
                    r.x += wa * ov.x;
                    r.y += wa * ov.y;
                    r.z += wa * ov.z;
                    r.w += wa * ov.w;
                }
                orow_p[d4] = r;
            }
        if (g == 0) a.lse[orow + qi] = lse_n;
    }
}

// The state of no block: o = 0, lse = -inf.
__global__ __launch_bounds__(256) void attn_empty_state(float* o, float* lse, int64_t rows, int64_t d)
{
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < rows * d; e += int64_t(gridDim.x) * 256) {
        o[e] = 0.f;
        if (e % d == 0) lse[e / d] = -__builtin_inff();
    }
}

template <int D>
hipError_t launch_d(int64_t bh, int64_t sq, int64_t sk, float scale, const void* q, const void* k, const void* v,
                    float* o, float* lse, bool first, hipStream_t s)
{
    using C = AttnCfg<D>;
    AttnArgs a{};
    a.q = static_cast<const char*>(q);
    a.k = static_cast<const char*>(k);
    a.v = static_cast<const char*>(v);
    a.o = o;
    a.lse = lse;
    a.sq = int32_t(sq);
    a.sk = int32_t(sk);
    a.nqt = int32_t((sq + C::QB - 1) / C::QB);
    a.nblocks = uint32_t(bh * a.nqt);
    a.c2 = scale * kLog2e;
    a.first = first ? 1 : 0;
    auto fn = &attn_block<D>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       C::LDS);
    if (e != hipSuccess) return e;
    void* args[] = {&a};
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(a.nblocks), dim3(256), args, C::LDS, s);
}

}  // namespace

hipError_t launch_attn_block(int64_t bh, int64_t sq, int64_t sk, int64_t d, float scale, const void* q, const void* k,
                             const void* v, float* o, float* lse, bool first, hipStream_t s)
{
    if (d != 64 && d != 128) return hipErrorNotSupported;
    // 32-bit key offsets within a (batch, head) matrix; grid below 2^31
    if (sq >= (int64_t(1) << 30) || sk * d * 2 >= (int64_t(1) << 32) - 64) return hipErrorNotSupported;
    if (bh * ((sq + 255) / 256) >= (int64_t(1) << 31)) return hipErrorNotSupported;
    for (const void* p : {q, k, v}) if (reinterpret_cast<uintptr_t>(p) % 16 != 0) return hipErrorNotSupported;
    if (reinterpret_cast<uintptr_t>(o) % 16 != 0) return hipErrorNotSupported;
    if (bh * sq == 0) return hipSuccess;
    if (sk == 0) {
        if (!first) return hipSuccess;  // merging an empty block changes nothing
        const int64_t total = bh * sq * d;
        const unsigned grid = unsigned(std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 4096)));
        hipLaunchKernelGGL(attn_empty_state, dim3(grid), dim3(256), 0, s, o, lse, bh * sq, d);
        return hipGetLastError();
    }
    return d == 64 ? launch_d<64>(bh, sq, sk, scale, q, k, v, o, lse, first, s)
                   : launch_d<128>(bh, sq, sk, scale, q, k, v, o, lse, first, s);
}

}  // namespace shardconv
