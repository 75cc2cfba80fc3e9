// One block step of ring attention (the paper's first benchmark, section
// "Performance Benchmarks", subsection "Ring Attention"): the local queries
// attend to the key/value block the device holds, and the result is merged in
// log space into the running (output, log-normaliser) state.
//
// Flash-style forward on v_mfma_f32_32x32x16_bf16, per (batch*head, 256-query
// tile) workgroup of eight waves, each wave owning one 32-query tile; the two
// waves of a SIMD (w and w + 4) take turns: while one runs its MFMAs, the other
// runs its softmax VALU work (below, the key loop):
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
//    buffered, 16-byte units XOR-swizzled by key so that the fragment reads
//    spread over the banks; keys past the block end load as zero and are
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
    static constexpr int NW = 8;               // waves: group A (0-3) and group B (4-7)
    static constexpr int THREADS = 64 * NW;
    static constexpr int QB = NW * 32;         // queries per workgroup, 32 per wave
    static constexpr int KB = 32;              // keys per block
    static constexpr int NC = D / 16;          // MFMA K steps over the head dim
    static constexpr int NDT = D / 32;         // 32-row head-dim tiles of O^T
    static constexpr int ROWB = D * 2;         // bytes per key row
    static constexpr int UPR = ROWB / 16;      // 16-byte units per row
    static constexpr int KV_BYTES = KB * ROWB; // one K or V block
    static constexpr int NLDW = KV_BYTES / 1024;  // wave loads (64 lanes x 16 B) per matrix per block
    static constexpr int STAGE = 2 * KV_BYTES;    // K block, then V block
    static constexpr int LDS = 2 * STAGE;         // double buffered
    static constexpr int PRE = 4;                 // fragment reads issued ahead, in (K, V, V) triples
    static_assert(D == 64 || D == 128, "head dim 64 or 128");
    static_assert(NC == 2 * NDT, "one O^T MFMA per score MFMA");
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

template <int B>
using ic = std::integral_constant<int, B>;

// kinds of iteration k of the key loop (see the kernel)
enum { kFirst, kFirstLast, kMid, kLast, kFinal };

template <int D>
__global__ __launch_bounds__(512, 1) void attn_block(AttnArgs a)
{
    using C = AttnCfg<D>;
    extern __shared__ uint4 lds4[];
    char* lds = reinterpret_cast<char*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    // a workgroup's waves w and w + 4 share a SIMD; the two groups run the
    // score/O^T MFMAs and the softmax VALU work in alternation (below)
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const bool grp_a = wv < 4;
    const uint32_t L = uint32_t(xcd_remap(blockIdx.x, gridDim.x));
    const uint32_t bh = L / uint32_t(a.nqt), qt = L - bh * uint32_t(a.nqt);
    const int qi = int(qt) * C::QB + wave * 32 + ln;  // this lane's query

    // Q^T fragments (B operand of S^T): lane (g, n) holds q[n][16c + 8g .. + 8]
    uint4 qf[C::NC];
    {
        const uint4* qm = reinterpret_cast<const uint4*>(a.q + int64_t(bh) * a.sq * C::ROWB);
#pragma unroll
        for (int c = 0; c < C::NC; ++c)
            qf[c] = qi < a.sq ? qm[int64_t(qi) * C::UPR + 2 * c + g] : make_uint4(0, 0, 0, 0);
    }

    // staging: wave load i fills LDS bytes [1024 i, 1024 i + 1024) of a block,
    // lane l bytes 1024 i + 16 l: key row r, slot s; it reads unit
    // k_slot/v_slot^-1 of that key. Iteration k stages K of block k + 1 and V of
    // block k (V runs one block behind: iteration k multiplies the probabilities
    // of block k - 1); blocks past the end load as zero.
    const int64_t kv_bytes = int64_t(a.sk) * C::ROWB;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.k) + int64_t(bh) * kv_bytes, short(0), int(uint32_t(kv_bytes)), 0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.v) + int64_t(bh) * kv_bytes, short(0), int(uint32_t(kv_bytes)), 0x00020000);
    auto stage = [&](int kbk, int kbv, int buf) {
        for (int i = wv; i < C::NLDW; i += C::NW) {
            char* dst = lds + buf * C::STAGE + i * 1024;
            const int byte = i * 1024 + lane * 16;
            const int r = byte / C::ROWB, sl = (byte % C::ROWB) / 16;
            const int kk = kbk * C::KB + r, kv = kbv * C::KB + r;
            const uint32_t ku = uint32_t(kk) * C::ROWB + uint32_t(k_slot<D>(r, sl)) * 16;
            const uint32_t vu = uint32_t(kv) * C::ROWB + uint32_t(v_slot(r, sl)) * 16;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, SC_LDSA(dst), 16, kbk >= 0 && kk < a.sk ? ku : 0xFFFFFFC0u,
                                                     0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, SC_LDSA(dst + C::KV_BYTES), 16,
                                                     kbv >= 0 && kv < a.sk ? vu : 0xFFFFFFC0u, 0, 0, 0);
        }
    };

    f32x16_a o[C::NDT];
    float m = -__builtin_inff(), l = 0.f, alpha = 1.f;
    bool resc = false;
#pragma unroll
    for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;

    // fragment read addresses in buffer 0 (buffer 1 is an immediate offset
    // away). K: lane (g, key n) reads unit 2c + g of its key, slot
    // (2c + g) ^ (n % UPR) = 2 (c ^ zh) + (g ^ zl) with zh = (n % UPR) / 2, zl = n % 2.
    const uint32_t lds0 = lds_addr(lds);
    const int zk = ln & (C::UPR - 1);
    uint32_t kad[C::NC];
#pragma unroll
    for (int c = 0; c < C::NC; ++c)
        kad[c] = lds0 + uint32_t(ln * C::ROWB + 16 * (g ^ (zk & 1))) + 32u * (uint32_t(c) ^ uint32_t(zk >> 1));
    // V^T: within a 16-lane group G, lane i addresses key row 16c + 8h + 4(G/2) + i/4
    // at head-dim columns 32dt + 16(G%2) + 4(i%4): unit 4dt + x (x < 4), slot
    // (4dt + x) ^ 2(i/4) = 4 (dt ^ yb) + (x ^ 2 y1) with yb = i/8, y1 = (i/4) % 2.
    // The dt part is an immediate offset; yb moves even dt by +64 B, odd dt by -64.
    const int G = lane >> 4, ii = lane & 15;
    const int vx = 2 * (G & 1) + ((ii & 3) >> 1), vy1 = (ii >> 2) & 1, vyb = ii >> 3;
    const uint32_t vcom =
        lds0 + uint32_t((4 * (G >> 1) + (ii >> 2)) * C::ROWB + 16 * (vx ^ (2 * vy1)) + 8 * (ii & 1));
    const uint32_t ve0 = vcom + 64u * uint32_t(vyb), vo0 = vcom - 64u * uint32_t(vyb);
    const int nkb = (a.sk + C::KB - 1) / C::KB;

    f32x16_a sc;            // scores of the block between its MFMA and VALU phases
    uint32_t pn[2][4];      // its probabilities, bf16, as the O^T MFMAs' B operand

    // MFMA phase of block k (buffer BUF = k % 2): the score MFMAs of block k
    // (S^T = K Q^T, M = 32 keys, N = 32 queries) alternating with the O^T MFMAs
    // of block k - 1 (O^T = V^T P^T, M = 32 head-dim rows, K = 32 keys in two
    // steps c), which take the probabilities as the B operand with no data
    // movement: the MFMA's K slots of lane half g are the keys that lane holds
    // (16c + 4g + 0..3 and 16c + 8 + 4g + 0..3), and V^T is read in that key
    // order with ds_read_b64_tr_b16. Fragment reads run PRE (K, V, V) triples
    // ahead of the MFMAs, with explicit waits (LDS operations complete in order).
    auto mfma_phase = [&](auto buf_c, auto s_c, auto pv_c) {
        constexpr int BUF = decltype(buf_c)::value;
        constexpr bool DO_S = decltype(s_c)::value, DO_PV = decltype(pv_c)::value;
        if (DO_PV && resc) {
#pragma unroll
            for (int dt = 0; dt < C::NDT; ++dt)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
        }
        lds_u32x4 kf[C::NC];
        uint2 vr[C::NC][2];
        auto issue = [&](auto j_c) {
            constexpr int j = decltype(j_c)::value, c = j / C::NDT, dt = j % C::NDT;
            kf[j] = lds_read_b128<BUF * C::STAGE>(kad[j]);
            constexpr int voff = BUF * C::STAGE + C::KV_BYTES + 16 * c * C::ROWB + 64 * dt;
            vr[j][0] = lds_read_tr16_b64<voff>((dt & 1) ? vo0 : ve0);
            vr[j][1] = lds_read_tr16_b64<voff + 8 * C::ROWB>((dt & 1) ? vo0 : ve0);
        };
        static_for<(C::PRE < C::NC ? C::PRE : C::NC)>(issue);
        static_for<C::NC>([&](auto j_c) {
            constexpr int j = decltype(j_c)::value, c = j / C::NDT, dt = j % C::NDT;
            constexpr int ahead = (C::NC - j < C::PRE ? C::NC - j : C::PRE);  // triples issued from j on
            lds_wait<3 * ahead - 1>();
            lds_ready(kf[j]);
            if (DO_S) {
                const f32x16_a cin = j == 0 ? f32x16_a{} : sc;
                sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_a, kf[j]),
                                                             __builtin_bit_cast(bf16x8_a, qf[j]), cin, 0, 0, 0);
            }
            lds_wait<3 * ahead - 3>();
            lds_ready(vr[j][0]);
            lds_ready(vr[j][1]);
            if (DO_PV) {
                const uint4 af = make_uint4(vr[j][0].x, vr[j][0].y, vr[j][1].x, vr[j][1].y);
                const uint4 bf = make_uint4(pn[c][0], pn[c][1], pn[c][2], pn[c][3]);
                o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_a, af),
                                                                __builtin_bit_cast(bf16x8_a, bf), o[dt], 0, 0, 0);
            }
            if constexpr (j + C::PRE < C::NC) issue(ic<j + C::PRE>{});
        });
    };

    // VALU phase of block k: masking (last block only), the row max against the
    // lazily moved reference (base 2, scores scaled by scale * log2 e), the
    // exponentials, their row sum into l and their bf16 rounding into pn. A
    // query's statistics live in one lane pair (g = 0, 1), joined by one
    // v_permlane32_swap. The reference max moves only when a block's scores
    // exceed it by more than 2^kSlack; alpha then rescales l here and O at the
    // start of the next MFMA phase.
    auto valu_phase = [&](int k, auto mask_c) {
        if (decltype(mask_c)::value) {
            const int kleft = a.sk - k * C::KB;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (8 * (r >> 2) + 4 * g + (r & 3) >= kleft) sc[r] = -__builtin_inff();
        }
        float v = fmaxf(sc[0], sc[1]);
#pragma unroll
        for (int r = 2; r < 16; r += 2) v = fmaxf(fmaxf(v, sc[r]), sc[r + 1]);
        {
            const uint32_t u = __float_as_uint(v);
            const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
            v = fmaxf(v, __uint_as_float(g ? p[0] : p[1])) * a.c2;
        }
        // the reference max moves for every lane when any lane needs it to
        resc = __builtin_amdgcn_ballot_w64(v > m + kSlack) != 0;
        const float mn = resc ? fmaxf(m, v) : m;
        alpha = __builtin_amdgcn_exp2f(m - mn);
        m = mn;
        float x[16];
        float sum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            x[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[r], a.c2, -m));
            sum += x[r];
        }
        const uint32_t u = __float_as_uint(sum);
        const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        l = l * alpha + sum + __uint_as_float(g ? p[0] : p[1]);
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bf16x2_a pk = {__bf16(x[8 * c + 2 * e]), __bf16(x[8 * c + 2 * e + 1])};
                pn[c][e] = __builtin_bit_cast(uint32_t, pk);
            }
    };

    // Iteration k: group A runs the MFMA phase of block k, then the VALU phase
    // of block k; group B the VALU phase of block k - 1, then the MFMA phase of
    // block k. So while one wave of a SIMD multiplies, the other does its
    // softmax work; a wave raises its priority for its MFMA phase, so that the
    // matrix core is fed first. Both phases read the buffer staged one
    // iteration earlier; the iteration ends with every wave's staging loads
    // landed and its LDS reads done, then a barrier, after which that buffer
    // may be refilled.
    // The whole key loop is written once per group (no joins of the two
    // groups' register state inside it); the barriers pair up across groups.
    auto run = [&](auto grp_c) {
        constexpr bool A = decltype(grp_c)::value;
        auto iteration = [&](int k, auto buf_c, auto kind_c) {
            constexpr int KIND = decltype(kind_c)::value;
            constexpr bool first = KIND == kFirst || KIND == kFirstLast, final = KIND == kFinal;
            using S = std::integral_constant<bool, !final>;
            using PV = std::integral_constant<bool, !first>;
            constexpr int BUF = decltype(buf_c)::value;
            if (!final) stage(k + 1 < nkb ? k + 1 : -1, k, BUF ^ 1);
            if constexpr (A) {
                __builtin_amdgcn_s_setprio(1);
                mfma_phase(buf_c, S{}, PV{});
                __builtin_amdgcn_s_setprio(0);
                if constexpr (!final)
                    valu_phase(k, std::integral_constant<bool, KIND == kFirstLast || KIND == kLast>{});
            } else {
                if constexpr (!first) valu_phase(k - 1, std::integral_constant<bool, final>{});
                __builtin_amdgcn_s_setprio(1);
                mfma_phase(buf_c, S{}, PV{});
                __builtin_amdgcn_s_setprio(0);
            }
            wait_vm_barrier<0>();
        };
        if (nkb == 1) {
            iteration(0, ic<0>{}, ic<kFirstLast>{});
            iteration(1, ic<1>{}, ic<kFinal>{});
        } else {
            iteration(0, ic<0>{}, ic<kFirst>{});
            int k = 1;
            for (; k + 2 < nkb; k += 2) {
                iteration(k, ic<1>{}, ic<kMid>{});
                iteration(k + 1, ic<0>{}, ic<kMid>{});
            }
            if (k + 1 < nkb) {
                iteration(k, ic<1>{}, ic<kMid>{});
                iteration(k + 1, ic<0>{}, ic<kLast>{});
                iteration(k + 2, ic<1>{}, ic<kFinal>{});
            } else {
                iteration(k, ic<1>{}, ic<kLast>{});
                iteration(k + 1, ic<0>{}, ic<kFinal>{});
            }
        }
    };
    stage(0, -1, 0);
    wait_vm_barrier<0>();
    if (grp_a)
        run(std::true_type{});
    else
        run(std::false_type{});

    // epilogue: lane (g, n) holds head-dim rows 32dt + 8j + 4g + e (e < 4) of
    // query qi; merge with the stored state
    if (qi >= a.sq) return;
    const int64_t orow = int64_t(bh) * a.sq;
    const float lse_b = (m + __builtin_amdgcn_logf(l)) * kLn2;
    const float inv = 1.f / l;
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
            r.x = o[dt][4 * j + 0] * wb;
            r.y = o[dt][4 * j + 1] * wb;
            r.z = o[dt][4 * j + 2] * wb;
            r.w = o[dt][4 * j + 3] * wb;
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
    return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(a.nblocks), dim3(C::THREADS), args, C::LDS, s);
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
