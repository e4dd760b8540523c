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
// (tcu_probe_lds) the LDS read rate of the products' two fragment reads, a
// fourth (tcu_probe_dma) the rate of direct global -> LDS loads, and a
// fifth (tcu_probe_pingpong) the full-tile product's two-group phase
// structure with its parts added one at a time.
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
// 512 bytes per instruction with ds_read_b64_tr_b16 (kKind 1) or
// ds_read_b64_tr_b8 (kKind 2; 64 lanes x 8 contiguous bytes each), 16
// instructions per round over a 64 KiB region, the
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
        const u32x2 v = kKind == 1 ? lds_read_tr16(s + off + 8 * lane) : lds_read_tr8(s + off + 8 * lane);
        acc[0] ^= v[0];
        acc[1] ^= v[1];
      }
    }
  }
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}


// DMA-rate probe: every wave of a workgroup (4, 8 or 16 waves, one per CU)
// issues 4 direct global -> LDS loads of 1 KiB (global_load_lds_dwordx4)
// per round from its own 4 KiB window of `src` (cache-resident after the
// first round) into its own 4 KiB of LDS, keeping 3 rounds in flight.
__global__ __launch_bounds__(1024) void dma_probe_kernel(const unsigned char *__restrict__ src,
                                                         unsigned *__restrict__ out, int64_t iters) {
  __shared__ __attribute__((aligned(1024))) unsigned char s[65536];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // window: < 128 windows of 4 KiB (512 KiB of src)
  const unsigned goff = (unsigned)((((int)blockIdx.x & 7) * 16 + w) * 4096 + 16 * lane);
  const unsigned dst = lds_addr(s) + w * 4096;
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 4; ++k) dma_lds16_saddr(src, goff + k * 1024, dst + k * 1024);
    asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  out[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = ((const unsigned *)s)[threadIdx.x & 16383];
}

// Ping-pong skeleton: the full-tile product's phase structure on one
// workgroup of 8 waves per CU (group 0 = waves 0-3, group 1 = waves 4-7,
// one wave of each group per SIMD), the 32 products of a phase from
// registers, with the other group's work added one part at a time:
//   kMode 0: no ping-pong -- every wave issues products, no barriers;
//   kMode 1: ping-pong -- one group's products per phase, a barrier
//            between phases (raised issue priority while computing);
//   kMode 2: + the other group's fragment reads per phase (8 ds_read_b128
//            and 8 ds_read_b64_tr_b16 per wave, waited before the barrier);
//   kMode 3: + after the reads its 4 direct global -> LDS loads of 1 KiB
//            per wave, 3 phases kept in flight (the product's phase);
//   kMode 4: the loads without the reads.
// Per launch every SIMD issues 64 * iters products (32 per wave and round
// in kMode 0, 32 per phase and two phases per round otherwise).  The
// operands are random bfloat16 values, as in the product's workloads.
constexpr int kPingLds = 65536;
template <int kMode>
__device__ __forceinline__ void ping_side(u32x4 (&xf)[kFM], u32x4 (&wf)[kFN], unsigned char *lds,
                                          int grp, int q, int lane, int64_t it,
                                          const unsigned char *src) {
  if constexpr (kMode == 2 || kMode == 3) {
    const int flip = (int)(it & 1);
    const unsigned char *pa = lds + grp * 8192 + ((16 * lane) ^ (16 * flip));
#pragma unroll
    for (int i = 0; i < kFM; ++i) xf[i] = *(const u32x4 *)(pa + i * 1024);
    const unsigned char *pb = lds + 16384 + q * 4096 + ((8 * lane) ^ (8 * flip));
#pragma unroll
    for (int j = 0; j < kFN; ++j) {
      const u32x2 lo = lds_read_tr16(pb + j * 1024);
      const u32x2 hi = lds_read_tr16(pb + j * 1024 + 512);
      wf[j] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
  }
  if constexpr (kMode == 3 || kMode == 4) {
    // 64 blocks of 16 KiB in a 1 MiB source, each CU at its own offset
    const unsigned goff =
        (unsigned)((((int)blockIdx.x * 7 + (int)it) & 63) * 16384 + q * 4096 + 16 * lane);
    const unsigned dst = lds_addr(lds) + 32768 + q * 4096;
#pragma unroll
    for (int k = 0; k < 4; ++k) dma_lds16_saddr(src, goff + k * 1024, dst + k * 1024);
    asm volatile("s_waitcnt vmcnt(12) lgkmcnt(0)" ::: "memory");
  } else if constexpr (kMode == 2) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

template <int kMode>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2))) void
pingpong_probe_kernel(const u32x4 *__restrict__ ops, const unsigned char *__restrict__ src,
                      int64_t iters, unsigned *__restrict__ out) {
  extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = w >> 2, q = w & 3;
  // the first 32 KiB of LDS: this workgroup's operand words
  for (int i = threadIdx.x; i < 2048; i += 512)
    ((u32x4 *)lds)[i] = ops[(int64_t)blockIdx.x * 2048 + i];
  __syncthreads();
  u32x4 xf[kFM], wf[kFN];
#pragma unroll
  for (int i = 0; i < kFM; ++i) xf[i] = ((const u32x4 *)lds)[(threadIdx.x + 64 * i) & 2047];
#pragma unroll
  for (int i = 0; i < kFN; ++i) wf[i] = ((const u32x4 *)lds)[(threadIdx.x + 1024 + 64 * i) & 2047];
  f32x4 acc[kFN][kFM];
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto products = [&]() {
    if constexpr (kMode != 0) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn)
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm)
        acc[fn][fm] = mfma_k32(TCU_BF16_F32, wf[fn], xf[fm], acc[fn][fm]);
    if constexpr (kMode != 0) __builtin_amdgcn_s_setprio(0);
  };
  for (int64_t it = 0; it < iters; ++it) {
    if constexpr (kMode == 0) {
      products();
    } else {
      if (grp == 0) products();
      else ping_side<kMode>(xf, wf, lds, grp, q, lane, it, src);
      asm volatile("s_barrier" ::: "memory");
      if (grp == 1) products();
      else ping_side<kMode>(xf, wf, lds, grp, q, lane, it, src);
      asm volatile("s_barrier" ::: "memory");
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  unsigned h = 0;
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) h = h * 31u + __builtin_bit_cast(unsigned, acc[a][b][e]);
  out[(int64_t)blockIdx.x * 512 + threadIdx.x] = h;
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
// ds_read_b64_tr_b16, 2: ds_read_b64_tr_b8; threads 256, 512 or 1024.  Every wave issues
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
  else if (kind == 2)
    hipLaunchKernelGGL(tcu::lds_probe_kernel<2>, dim3(blocks), dim3(threads), 0, st, u, iters);
  else
    return -1;
  return hipGetLastError() == hipSuccess ? 0 : -6;
}

// src: 512 KiB or more of device memory; out: blocks * threads words
// (device); threads 256, 512 or 1024.  Every wave issues 4 * iters loads of
// 1 KiB into LDS.  Asynchronous on `stream`.  Returns 0, or -1 for bad
// arguments, -6 for a launch error.
extern "C" __attribute__((visibility("default"))) int tcu_probe_dma(const void *src, void *out,
                                                                    int64_t iters, int blocks,
                                                                    int threads, void *stream) {
  if (!src || !out || iters < 1 || blocks < 1 ||
      (threads != 256 && threads != 512 && threads != 1024))
    return -1;
  hipLaunchKernelGGL(tcu::dma_probe_kernel, dim3(blocks), dim3(threads), 0, (hipStream_t)stream,
                     static_cast<const unsigned char *>(src), static_cast<unsigned *>(out), iters);
  return hipGetLastError() == hipSuccess ? 0 : -6;
}

// ops: blocks * 2048 16-byte words (device); src: 1 MiB of device memory;
// out: blocks * 512 words (device); mode 0..4 as for pingpong_probe_kernel.
// Asynchronous on `stream`.  Returns 0, or -1 for bad arguments, -6 for a
// launch error.
extern "C" __attribute__((visibility("default"))) int tcu_probe_pingpong(int mode, const void *ops,
                                                                         const void *src, void *out,
                                                                         int64_t iters, int blocks,
                                                                         void *stream) {
  if (!ops || !src || !out || iters < 1 || blocks < 1 || mode < 0 || mode > 4) return -1;
  const auto *o = static_cast<const tcu::u32x4 *>(ops);
  const auto *g = static_cast<const unsigned char *>(src);
  auto *u = static_cast<unsigned *>(out);
  hipStream_t st = (hipStream_t)stream;
  switch (mode) {
#define TCU_PING(M)                                                                          \
  case M:                                                                                    \
    hipLaunchKernelGGL(tcu::pingpong_probe_kernel<M>, dim3(blocks), dim3(512), tcu::kPingLds, \
                       st, o, g, iters, u);                                                  \
    break;
    TCU_PING(0) TCU_PING(1) TCU_PING(2) TCU_PING(3) TCU_PING(4)
#undef TCU_PING
  }
  return hipGetLastError() == hipSuccess ? 0 : -6;
}
