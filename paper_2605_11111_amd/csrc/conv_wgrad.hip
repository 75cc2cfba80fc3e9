// Weight gradient launcher.
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace shardconv {

size_t generic_wgrad_workspace(const Tile3& t, const Conv3& cv);
hipError_t generic_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                              float* dw, void* ws, hipStream_t s);

size_t conv_wgrad_workspace(const Tile3& t, const Conv3& cv, shard_dtype_t dt)
{
    (void)dt;
    return generic_wgrad_workspace(t, cv);
}

hipError_t launch_conv_wgrad(const Tile3& t, const Conv3& cv, shard_dtype_t dt, const void* tile, const void* dy,
                             float* dw, void* ws, hipStream_t s)
{
    return generic_conv_wgrad(t, cv, dt, tile, dy, dw, ws, s);
}

}  // namespace shardconv
