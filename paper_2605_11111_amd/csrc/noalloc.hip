// shard_conv_fwd without a caller-provided workspace: the forward convolution's
// only scratch (the weights laid out in MFMA B-fragment order) lives in a
// file-scope device array, one copy per GPU, for callers that cannot allocate
// (code under graph capture, tight serving loops).
#include <mutex>

#include "internal.h"

namespace shardconv {
namespace {

// Upper bound of the weight-fragment scratch: 4 MiB holds the fragments of
// every workload shape of this library (the largest, 64 -> 128 channels at
// 3 x 3 x 3 in binary32, needs 864 KiB).
constexpr size_t kScratchBytes = size_t(4) << 20;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each device, looked up once per device with
// that device current (host code never passes the array's name itself).
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

hipError_t scratch_ptr(void** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return hipSuccess;
}

}  // namespace

size_t conv_fwd_noalloc_limit() { return kScratchBytes; }

hipError_t launch_conv_fwd_noalloc(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile,
                                   const void* w, void* y, hipStream_t s)
{
    void* ws = nullptr;
    const hipError_t e = scratch_ptr(&ws);
    if (e != hipSuccess) return e;
    return launch_conv_fwd(t, cv, dt, tile, w, y, ws, s);
}

}  // namespace shardconv
