// Entry points of the thread-per-product kernels (gtp_small.hip) beyond the
// launchers every kernel family shares (gtp_device.hpp).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gtp {

// Both input gradients of an equal-degree product L1 = L2 = Lout = L (1..7)
// in one launch: dx1 = P_L(GTP(dy, x2)), dx2 = P_L(GTP(dy, x1)) for n
// products (dy, dx1, dx2 fp32 rows of (L + 1)^2; x1, x2 rows of input type
// it, fp32 or bf16).  *supported = false for other degrees or types.
hipError_t launch_bwd_small(int L, const float* dy, const void* x1, const void* x2, int it, int64_t n, float* dx1,
                            float* dx2, hipStream_t s, bool* supported);

}  // namespace gtp
