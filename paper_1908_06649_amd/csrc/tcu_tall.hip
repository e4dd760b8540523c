// The native tensor-unit call of the (m,l)-TCU model (Section 3, model
// definition): C (n x s) = A (n x s) * B (s x s), for s = sqrt(m) in {16, 32}.
//
// The model's third property ("asymmetric behavior") says the unit first
// loads the weights B and then streams the n rows of A through it in chunks
// of sqrt(m) rows.  On gfx950 that maps onto one wavefront per stream of
// 16-row chunks:
//   * each wave reads B once, into the registers that feed the matrix core
//     as its row operand (B transposed), and keeps it there for the whole
//     call -- the weights stay in the unit;
//   * a chunk of 16 rows of A is one 16-byte (or 8-byte) load per lane, so a
//     wave's load covers 16 consecutive rows, i.e. a contiguous block of
//     memory; the chunk is the matrix core's column operand;
//   * the product is computed as C^T = B^T A^T, so every lane ends up holding
//     consecutive output columns of one row of C and the store is again a
//     contiguous block per wave;
//   * the grid is persistent: up to 16 workgroups per compute unit walk the
//     chunks with a grid stride, each wave keeping U chunk loads in flight;
//   * A is read and C written with non-temporal (streaming) accesses: each
//     byte is touched once, and keeping it out of the caches' normal
//     replacement measurably raises the achieved HBM bandwidth.
// For very tall A the call is bound by HBM bandwidth (n*s inputs read and
// n*s outputs written, against 2*n*s^2 flops); the matrix core keeps the
// arithmetic off the critical path.
#include "tcu_device.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kTallThreads = 256;  // 4 waves per workgroup

// Output column held by lane row m of weight block h when s = 32: the two
// 16-column blocks interleave in groups of 4 so that lane group g ends up
// with the 8 consecutive output columns 8g .. 8g+7.
__device__ __forceinline__ int col32(int m, int h) { return 8 * (m >> 2) + 4 * h + (m & 3); }

// 32-bit outputs: add the stored values (accumulating form, int32 with
// two's-complement wrap-around) to the fresh block d, as raw words.
template <int DT, typename Acc>
__device__ __forceinline__ u32x4 add_stored(Acc d, const u32x4 *p) {
  const u32x4 o = __builtin_nontemporal_load(p);
  if constexpr (DT == TCU_I8_I32)
    return bitcast<u32x4>(d) + o;
  else
    return bitcast<u32x4>(d + bitcast<f32x4>(o));
}

// bfloat16 outputs: 2*W values, the pairs (v[2i], v[2i+1]) packed per word,
// with the stored values added first when accumulating.
template <int W>
__device__ __forceinline__ void pack_out(const float *v, unsigned *words, const unsigned *old) {
#pragma unroll
  for (int i = 0; i < W; ++i) {
    float lo = v[2 * i], hi = v[2 * i + 1];
    if (old) {
      lo += bf16_to_f32(old[i] & 0xffffu);
      hi += bf16_to_f32(old[i] >> 16);
    }
    words[i] = pack_bf16x2(lo, hi);
  }
}

template <int DT, int S, int U, bool kAcc>
__global__ __launch_bounds__(kTallThreads) void tall_kernel(const unsigned char *__restrict__ A,
                                                            int64_t n,
                                                            const unsigned char *__restrict__ B,
                                                            unsigned char *__restrict__ C,
                                                            int64_t ntiles) {
  constexpr bool kI8 = (DT == TCU_I8_I32);
  constexpr int IB = in_bytes(DT);
  constexpr int OB = out_bytes(DT);
  constexpr int kRowIn = S * IB;   // bytes per row of A
  constexpr int kRowOut = S * OB;  // bytes per row of C
  // Each lane's contracted run: 8 elements (s = 32, or int8 any s) or
  // 4 elements (16-bit inputs, s = 16).
  constexpr int kRun = (S == 16 && !kI8) ? 4 : 8;
  constexpr int kRunBytes = kRun * IB;  // 16 or 8
  constexpr int kBlocks = S / 16;       // 16-column output blocks

  const int lane = threadIdx.x & 63;
  const int r = lane & 15;  // row of the 16-row chunk handled by this lane
  const int g = lane >> 4;  // lane group: selects the contracted run
  // int8 with s = 16 uses the K = 32 instruction; lane groups 2, 3 carry zeros.
  const bool k_live = !(kI8 && S == 16) || g < 2;

  // ---- load the weights once (B transposed, matrix-core row operand) ----
  typedef typename std::conditional<kRunBytes == 16, u32x4, u32x2>::type Run;
  Run w[kBlocks];
#pragma unroll
  for (int h = 0; h < kBlocks; ++h) {
    const int j = (S == 32) ? col32(r, h) : r;
    unsigned words[kRunBytes / 4];
#pragma unroll
    for (int q = 0; q < kRunBytes / 4; ++q) words[q] = 0;
    if (k_live) {
#pragma unroll
      for (int i = 0; i < kRun; ++i) {
        const int k = g * kRun + i;
        unsigned v;
        if (kI8)
          v = (unsigned)B[k * S + j];
        else
          v = (unsigned)((const unsigned short *)B)[k * S + j];
        words[(i * IB) / 4] |= v << (8 * ((i * IB) % 4));
      }
    }
    Run wv;
#pragma unroll
    for (int q = 0; q < kRunBytes / 4; ++q) wv[q] = words[q];
    w[h] = wv;
  }

  const int64_t wave = (int64_t)blockIdx.x * (kTallThreads / 64) + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * (kTallThreads / 64);

  for (int64_t t0 = wave * U; t0 < ntiles; t0 += nwaves * U) {
    Run x[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = (t0 + u) * 16 + r;
      ok[u] = row < n;
      Run z = {};
      x[u] = (ok[u] && k_live)
                 ? __builtin_nontemporal_load((const Run *)(A + row * kRowIn + g * kRunBytes))
                 : z;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = (t0 + u) * 16 + r;
      unsigned char *crow = C + row * kRowOut;
      if constexpr (kI8) {
        i32x4 d[kBlocks];
#pragma unroll
        for (int h = 0; h < kBlocks; ++h) d[h] = mfma_i8_k32(w[h], x[u], i32x4{0, 0, 0, 0});
        if (ok[u]) {
#pragma unroll
          for (int h = 0; h < kBlocks; ++h) {
            u32x4 *p = (u32x4 *)(crow + (S == 32 ? 32 * g + 16 * h : 16 * g));
            __builtin_nontemporal_store(kAcc ? add_stored<DT>(d[h], p) : bitcast<u32x4>(d[h]), p);
          }
        }
      } else {
        f32x4 d[kBlocks];
#pragma unroll
        for (int h = 0; h < kBlocks; ++h) {
          if constexpr (S == 32)
            d[h] = mfma_k32(DT, w[h], x[u], f32x4{0.f, 0.f, 0.f, 0.f});
          else
            d[h] = mfma_k16(DT, w[h], x[u], f32x4{0.f, 0.f, 0.f, 0.f});
        }
        if (ok[u]) {
          if constexpr (DT == TCU_BF16_BF16) {
            // Output columns 4*kBlocks*g .. +4*kBlocks-1 of the row, in order.
            float v[4 * kBlocks];
#pragma unroll
            for (int h = 0; h < kBlocks; ++h)
#pragma unroll
              for (int i = 0; i < 4; ++i) v[4 * h + i] = d[h][i];
            if constexpr (S == 32) {
              u32x4 *p = (u32x4 *)(crow + 16 * g);
              unsigned w[4], old[4];
              if (kAcc) {
                const u32x4 o = __builtin_nontemporal_load(p);
                for (int i = 0; i < 4; ++i) old[i] = o[i];
              }
              pack_out<4>(v, w, kAcc ? old : nullptr);
              __builtin_nontemporal_store(u32x4{w[0], w[1], w[2], w[3]}, p);
            } else {
              u32x2 *p = (u32x2 *)(crow + 8 * g);
              unsigned w[2], old[2];
              if (kAcc) {
                const u32x2 o = __builtin_nontemporal_load(p);
                old[0] = o[0];
                old[1] = o[1];
              }
              pack_out<2>(v, w, kAcc ? old : nullptr);
              __builtin_nontemporal_store(u32x2{w[0], w[1]}, p);
            }
          } else {
#pragma unroll
            for (int h = 0; h < kBlocks; ++h) {
              u32x4 *p = (u32x4 *)(crow + (S == 32 ? 32 * g + 16 * h : 16 * g));
              __builtin_nontemporal_store(kAcc ? add_stored<DT>(d[h], p) : bitcast<u32x4>(d[h]), p);
            }
          }
        }
      }
    }
  }
}

template <int DT, int S>
hipError_t launch_one(const void *A, int64_t n, const void *B, void *C, bool accum,
                      hipStream_t stream, int num_cus) {
  constexpr int U = 4;
  const int64_t ntiles = (n + 15) / 16;
  const int64_t want = (ntiles + 4 * U - 1) / (4 * U);
  const int64_t cap = (int64_t)num_cus * 16;
  const int blocks = (int)(want < cap ? want : cap);
  if (accum)
    hipLaunchKernelGGL((tall_kernel<DT, S, U, true>), dim3(blocks), dim3(kTallThreads), 0,
                       stream, (const unsigned char *)A, n, (const unsigned char *)B,
                       (unsigned char *)C, ntiles);
  else
    hipLaunchKernelGGL((tall_kernel<DT, S, U, false>), dim3(blocks), dim3(kTallThreads), 0,
                       stream, (const unsigned char *)A, n, (const unsigned char *)B,
                       (unsigned char *)C, ntiles);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tall(int dtype, int s, const void *A, int64_t n, const void *B, void *C,
                       bool accum, hipStream_t stream, int num_cus) {
  switch (dtype * 2 + (s == 32 ? 1 : 0)) {
    case TCU_F16_F32 * 2 + 0: return launch_one<TCU_F16_F32, 16>(A, n, B, C, accum, stream, num_cus);
    case TCU_F16_F32 * 2 + 1: return launch_one<TCU_F16_F32, 32>(A, n, B, C, accum, stream, num_cus);
    case TCU_BF16_F32 * 2 + 0: return launch_one<TCU_BF16_F32, 16>(A, n, B, C, accum, stream, num_cus);
    case TCU_BF16_F32 * 2 + 1: return launch_one<TCU_BF16_F32, 32>(A, n, B, C, accum, stream, num_cus);
    case TCU_BF16_BF16 * 2 + 0: return launch_one<TCU_BF16_BF16, 16>(A, n, B, C, accum, stream, num_cus);
    case TCU_BF16_BF16 * 2 + 1: return launch_one<TCU_BF16_BF16, 32>(A, n, B, C, accum, stream, num_cus);
    case TCU_I8_I32 * 2 + 0: return launch_one<TCU_I8_I32, 16>(A, n, B, C, accum, stream, num_cus);
    case TCU_I8_I32 * 2 + 1: return launch_one<TCU_I8_I32, 32>(A, n, B, C, accum, stream, num_cus);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcu
