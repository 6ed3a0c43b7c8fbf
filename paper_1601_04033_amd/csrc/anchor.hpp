// Launcher of the bandwidth anchor (a diagnostic, apart from the method's
// kernels declared in kernels.hpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fasgd {

// dst[0, n) = src[0, n), 16-byte aligned arrays.
hipError_t launch_copy_anchor(const float* src, float* dst, int64_t n, hipStream_t s);

}  // namespace fasgd
