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
//
// A second probe (tcu_probe_overlap) measures whether binary32 vector ALU
// work runs while the matrix core works: interleaved in one wave's
// instruction stream, or issued by other waves on the same SIMD; a third
// (tcu_probe_lds) the LDS read rate of the products' two fragment reads.
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

// Overlap probe: can binary32 vector ALU work run while the matrix core
// works, and from which waves?  Every lane keeps 8 independent binary32
// chains (v = v * c1 + c2) beside 8 independent bfloat16 accumulators.
//   kMode 0 (one wave does both): each wave issues 32 matrix-core
//     instructions per round, each followed by NV vector FMAs that do not
//     depend on it (the order held by scheduling barriers);
//   kMode 1 (separate waves): waves 0-3 issue the 32 matrix-core
//     instructions per round, waves 4-7 -- on the same four SIMDs -- 32 * NV
//     vector FMAs per round;
//   kMode 2: only waves 0-3 (matrix core) work; kMode 3: only waves 4-7
//     (vector ALU) work; the other waves write their word and exit.
template <int kMode, int NV>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2))) void
overlap_probe_kernel(const u32x4 *__restrict__ ops, int64_t iters, unsigned *__restrict__ out) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool mfma_wave = kMode == 0 || ((kMode == 1 || kMode == 2) && w < 4);
  const bool valu_wave = kMode == 0 || ((kMode == 1 || kMode == 3) && w >= 4);
  const u32x4 *p = ops + t * 3;
  const u32x4 xw = p[0], ww = p[1], vw = p[2];
  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = __builtin_bit_cast(float, (vw[i & 3] >> (i & 4)) & 0x3f7fffffu);
  const float c1 = 0.999f, c2 = 1e-3f;
  if (mfma_wave && valu_wave) {
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        acc[j & 7] = mfma_k32(TCU_BF16_F32, ww, xw, acc[j & 7]);
#pragma unroll
        for (int i = 0; i < NV; ++i) v[(j * NV + i) & 7] = __builtin_fmaf(v[(j * NV + i) & 7], c1, c2);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (NV > 0) __builtin_amdgcn_sched_group_barrier(0x002, NV, 0);
      }
    }
  } else if (mfma_wave) {
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 32; ++j) acc[j & 7] = mfma_k32(TCU_BF16_F32, ww, xw, acc[j & 7]);
    }
  } else if (valu_wave) {
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 32 * NV; ++j) v[j & 7] = __builtin_fmaf(v[j & 7], c1, c2);
    }
  }
  unsigned h = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i)
    h = h * 31u + __builtin_bit_cast(unsigned, acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3] + v[i]);
  out[t] = h;
}

// LDS read-rate probe: every wave of a workgroup (4, 8 or 16 waves, one
// workgroup per CU) reads 1 KiB per instruction with
// ds_read_b128 (kKind 0; 64 lanes x 16 contiguous bytes, conflict-free) or
// 512 bytes per instruction with ds_read_b64_tr_b16 (kKind 1; 64 lanes x 8
// contiguous bytes), 16 instructions per round over a 64 KiB region, the
// offset moving every round so that no read can be hoisted; the values are
// folded into one word per lane.
template <int kKind>
__global__ __launch_bounds__(1024) void lds_probe_kernel(unsigned *__restrict__ out, int64_t iters) {
  __shared__ __attribute__((aligned(16))) unsigned char s[65536];
  for (int i = threadIdx.x; i < 65536 / 16; i += blockDim.x)
    ((u32x4 *)s)[i] = u32x4{(unsigned)i, 1u, 2u, 3u};
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int off = ((w * 16 + j + (int)(it & 63)) & 63) * 1024;   // < 64 KiB
      if constexpr (kKind == 0) {
        acc ^= *(const u32x4 *)(s + off + 16 * lane);
      } else {
        const u32x2 v = lds_read_tr16(s + off + 8 * lane);
        acc[0] ^= v[0];
        acc[1] ^= v[1];
      }
    }
  }
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

template <int kMode>
hipError_t launch_overlap(int nv, const u32x4 *ops, int64_t iters, unsigned *out, int blocks,
                          hipStream_t stream) {
  switch (nv) {
#define TCU_OVL(N)                                                                          \
  case N:                                                                                  \
    hipLaunchKernelGGL((overlap_probe_kernel<kMode, N>), dim3(blocks), dim3(512), 0, stream, \
                       ops, iters, out);                                                   \
    break;
    TCU_OVL(0) TCU_OVL(1) TCU_OVL(2) TCU_OVL(3) TCU_OVL(4) TCU_OVL(6)
#undef TCU_OVL
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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

// ops: blocks * 512 * 3 16-byte words (device); out: blocks * 512 words
// (device).  mode 0..3 as for overlap_probe_kernel; nv in {0, 1, 2, 3, 4, 6}
// vector FMAs per matrix-core instruction.  Asynchronous on `stream`.
// Returns 0, or -1 for bad arguments, -6 for a launch error.
extern "C" __attribute__((visibility("default"))) int tcu_probe_overlap(int mode, int nv,
                                                                        const void *ops, void *out,
                                                                        int64_t iters, int blocks,
                                                                        void *stream) {
  if (!ops || !out || iters < 1 || blocks < 1 || mode < 0 || mode > 3) return -1;
  const auto *o = static_cast<const tcu::u32x4 *>(ops);
  auto *u = static_cast<unsigned *>(out);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e;
  switch (mode) {
    case 0: e = tcu::launch_overlap<0>(nv, o, iters, u, blocks, st); break;
    case 1: e = tcu::launch_overlap<1>(nv, o, iters, u, blocks, st); break;
    case 2: e = tcu::launch_overlap<2>(nv, o, iters, u, blocks, st); break;
    default: e = tcu::launch_overlap<3>(nv, o, iters, u, blocks, st); break;
  }
  if (e == hipErrorInvalidValue) return -1;
  return e == hipSuccess ? 0 : -6;
}

// out: blocks * threads words (device).  kind 0: ds_read_b128, 1:
// ds_read_b64_tr_b16; threads 256, 512 or 1024.  Every wave issues
// 16 * iters LDS read instructions.  Asynchronous on `stream`.  Returns 0,
// or -1 for bad arguments, -6 for a launch error.
extern "C" __attribute__((visibility("default"))) int tcu_probe_lds(int kind, void *out,
                                                                    int64_t iters, int blocks,
                                                                    int threads, void *stream) {
  if (!out || iters < 1 || blocks < 1 || (threads != 256 && threads != 512 && threads != 1024))
    return -1;
  auto *u = static_cast<unsigned *>(out);
  hipStream_t st = (hipStream_t)stream;
  if (kind == 0)
    hipLaunchKernelGGL(tcu::lds_probe_kernel<0>, dim3(blocks), dim3(threads), 0, st, u, iters);
  else if (kind == 1)
    hipLaunchKernelGGL(tcu::lds_probe_kernel<1>, dim3(blocks), dim3(threads), 0, st, u, iters);
  else
    return -1;
  return hipGetLastError() == hipSuccess ? 0 : -6;
}
