// Sustained bf16 matrix-instruction rate of the part: nothing but MFMAs in
// independent accumulation chains, the clock read at both ends. The part is
// power-limited under MFMA load and the power drawn depends on how much the
// operand bits toggle, so the kernel runs either on constant operands or on
// random ones that change from one instruction to the next.
#include <hip/hip_runtime.h>

#include "shardprobe.h"

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

constexpr int kChains = 4;
constexpr int kFrags = 4;  // operand fragments in rotation (random mode)

__device__ uint32_t mix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// roughly N(0, 1) bf16 values: a centred sum of four uniforms, scaled
__device__ bf16x8_t random_frag(uint32_t seed)
{
    bf16x8_t v;
    for (int i = 0; i < 8; ++i) {
        float u = 0.f;
        for (int k = 0; k < 4; ++k) u += float(mix32(seed * 64u + uint32_t(i * 4 + k)) & 0xffffu) * (1.f / 65536.f);
        v[i] = __bf16((u - 2.f) * 1.7f);
    }
    return v;
}

__global__ __launch_bounds__(256) void mfma_ceiling(int64_t iters, int32_t random, float* out, uint64_t* clk)
{
    bf16x8_t a[kFrags], b[kFrags];
    for (int j = 0; j < kFrags; ++j) {
        const uint32_t base = (blockIdx.x * 256u + threadIdx.x) * 2u * kFrags;
        if (random) {
            a[j] = random_frag(base + uint32_t(j));
            b[j] = random_frag(base + uint32_t(kFrags + j));
        } else {
            for (int i = 0; i < 8; ++i) {
                a[j][i] = __bf16(float(threadIdx.x + i) * 1e-3f);
                b[j][i] = __bf16(float(i + 1) * 1e-3f);
            }
        }
    }
    f32x16_t acc[kChains];
    for (int c = 0; c < kChains; ++c)
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    // kFrags instructions per chain per trip; the fragment indices are
    // compile-time constants (a runtime index into a register array would go
    // through scratch memory)
    for (int64_t it = 0; it < iters; it += kFrags) {
#pragma unroll
        for (int j = 0; j < kFrags; ++j)
#pragma unroll
            for (int c = 0; c < kChains; ++c)
                acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(c + j) % kFrags], b[(c + 2 * j + 1) % kFrags],
                                                                  acc[c], 0, 0, 0);
    }
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    float s = 0.f;
    for (int c = 0; c < kChains; ++c)
        for (int e = 0; e < 16; ++e) s += acc[c][e];
    out[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
    if (threadIdx.x == 0) {
        clk[2 * int64_t(blockIdx.x)] = t1 - t0;
        clk[2 * int64_t(blockIdx.x) + 1] = r1 - r0;
    }
}

}  // namespace

extern "C" int shard_probe_mfma_bf16(int64_t iters, int32_t blocks, int32_t random, float* out, uint64_t* clk,
                                     hipStream_t stream)
{
    if (iters < 1 || iters % kFrags != 0 || blocks < 1 || out == nullptr || clk == nullptr) return 1;
    hipLaunchKernelGGL(mfma_ceiling, dim3(unsigned(blocks)), dim3(256), 0, stream, iters, random, out, clk);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}
