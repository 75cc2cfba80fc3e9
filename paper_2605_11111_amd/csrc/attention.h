// Internal interface of the ring-attention block step (attention.hip).
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

namespace shardconv {

// One block step for q [bh][sq][d], k and v [bh][sk][d] (bf16) merged into the
// running state o [bh][sq][d], lse [bh][sq] (binary32); d is 64 or 128.
// Returns hipErrorNotSupported for shapes the kernel does not take.
hipError_t launch_attn_block(int64_t bh, int64_t sq, int64_t sk, int64_t d, float scale, const void* q, const void* k,
                             const void* v, float* o, float* lse, bool first, hipStream_t s);

}  // namespace shardconv
