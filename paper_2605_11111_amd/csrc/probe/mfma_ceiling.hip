// Sustained bf16 matrix-instruction rate of the part: nothing but MFMAs in
// independent accumulation chains, the clock read at both ends.
#include <hip/hip_runtime.h>

#include "shardprobe.h"

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

constexpr int kChains = 4;

__global__ __launch_bounds__(256) void mfma_ceiling(int64_t iters, float* out, uint64_t* clk)
{
    bf16x8_t a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = __bf16(float(threadIdx.x + i) * 1e-3f);
        b[i] = __bf16(float(i + 1) * 1e-3f);
    }
    f32x16_t acc[kChains];
    for (int c = 0; c < kChains; ++c)
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
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

extern "C" int shard_probe_mfma_bf16(int64_t iters, int32_t blocks, float* out, uint64_t* clk, hipStream_t stream)
{
    if (iters < 1 || blocks < 1 || out == nullptr || clk == nullptr) return 1;
    hipLaunchKernelGGL(mfma_ceiling, dim3(unsigned(blocks)), dim3(256), 0, stream, iters, out, clk);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}
