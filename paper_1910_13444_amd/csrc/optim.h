// Parameter update kernels of libpigan.so (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pigan {

// Adam on fp32 master weights; skip (device int or null) non-zero leaves
// every array unchanged.  c1 = 1/(1 - b1^t), c2 = 1/(1 - b2^t).
hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v, float lr, float b1, float b2,
                       float eps, float c1, float c2, const int32_t* skip, hipStream_t st);

}  // namespace pigan
