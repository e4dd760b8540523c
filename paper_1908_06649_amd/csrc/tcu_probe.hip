// Matrix-core ceiling probe for the benchmark (not part of the library's
// C ABI; built into its own libtcu_probe.so).
//
// It measures what the matrix cores sustain on this chip when they do
// nothing else: every wave of a persistent grid shaped like the full-tile
// product's (one workgroup of 8 waves per CU, two waves per SIMD) loads the
// operands of one of the product's phases -- 8 data and 4 weights
// fragments, 16 bytes per lane each -- once from memory, then issues `iters`
// rounds of the product's 32 matrix-core instructions on them from
// registers (16x16x32 bfloat16 into binary32, or 16x16x64 int8 into int32),
// and finally writes one sum of its accumulators per lane so that no work
// is dead.  No LDS, no further memory traffic, no barriers: the rate is
// bounded by the matrix cores and the chip's clock under the power limit,
// which depends on the operand values (the host passes random or constant
// data).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tcu_device.h"

namespace tcu {
namespace {

constexpr int kFM = 8, kFN = 4;   // the product's wave sub-tile: 32 blocks of 16 x 16

template <int DT>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2))) void
mfma_probe_kernel(const u32x4 *__restrict__ ops, int64_t iters, unsigned *__restrict__ out) {
  constexpr bool kI8 = DT == TCU_I8_I32;
  typedef typename std::conditional<kI8, i32x4, f32x4>::type Acc;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const u32x4 *p = ops + t * (kFM + kFN);
  u32x4 xf[kFM], wf[kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i) xf[i] = p[i];
#pragma unroll
  for (int i = 0; i < kFN; ++i) wf[i] = p[kFM + i];
  Acc acc[kFN][kFM];
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b) acc[a][b] = Acc{0, 0, 0, 0};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm) {
        if constexpr (kI8)
          acc[fn][fm] = mfma_i8_k64(wf[fn], xf[fm], acc[fn][fm]);
        else
          acc[fn][fm] = mfma_k32(DT, wf[fn], xf[fm], acc[fn][fm]);
      }
  }
  unsigned h = 0;
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) h = h * 31u + __builtin_bit_cast(unsigned, acc[a][b][e]);
  out[t] = h;
}

}  // namespace
}  // namespace tcu

// ops: blocks * 512 * 12 16-byte operand words (device); out: blocks * 512
// words (device).  dtype: TCU_BF16_F32 or TCU_I8_I32.  Asynchronous on
// `stream`.  Returns 0, or -1 for bad arguments, -6 for a launch error.
// Every wave issues 32 * iters matrix-core instructions.
extern "C" __attribute__((visibility("default"))) int tcu_probe_mfma(int dtype, const void *ops,
                                                                     void *out, int64_t iters,
                                                                     int blocks, void *stream) {
  if (!ops || !out || iters < 1 || blocks < 1) return -1;
  const auto *o = static_cast<const tcu::u32x4 *>(ops);
  auto *u = static_cast<unsigned *>(out);
  if (dtype == TCU_BF16_F32)
    hipLaunchKernelGGL((tcu::mfma_probe_kernel<TCU_BF16_F32>), dim3(blocks), dim3(512), 0,
                       (hipStream_t)stream, o, iters, u);
  else if (dtype == TCU_I8_I32)
    hipLaunchKernelGGL((tcu::mfma_probe_kernel<TCU_I8_I32>), dim3(blocks), dim3(512), 0,
                       (hipStream_t)stream, o, iters, u);
  else
    return -1;
  return hipGetLastError() == hipSuccess ? 0 : -6;
}
