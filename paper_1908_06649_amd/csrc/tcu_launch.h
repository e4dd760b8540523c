// Internal launchers behind the C ABI (host side).  Arguments are already
// validated by the ABI layer; these only pick a kernel instance and launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tcu {

// Native call: C (n x s) = A (n x s) * B (s x s) for s in {16, 32}.
hipError_t launch_tall(int dtype, int s, const void *A, int64_t n, const void *B, void *C,
                       hipStream_t stream, int num_cus);

// Blocked product of Theorem 2 fused into one launch: C (N x N) = A * B.
hipError_t launch_gemm(int dtype, const void *A, const void *B, void *C, int64_t N,
                       hipStream_t stream, int num_cus);

}  // namespace tcu
