// Transitive closure of a directed graph (Section 4.3, Theorem 5), in place
// on its n x n 0/1 adjacency matrix X (int8, row pitch ld).
//
// The section's blocked algorithm walks the pivot blocks k in order and, for
// each, closes the diagonal block (function A), updates the pivot block row
// (B) and block column (C) through it, and updates every other block with
// X_ij <- min(X_ij + X_ik X_kj, 1) (function D) -- plain multiplication and
// addition on the unit, clamped, which equals OR-of-ANDs because X_ij is
// disjoint from X_ik and X_kj.  D is the hot path (about n^2/m calls per
// pivot); it runs on the int8 matrix cores.
//
// Here the pivot band is Bk = 256 vertices (8 of the unit's 32-wide blocks
// at once): the diagonal 256 x 256 block is closed by the iterative
// algorithm itself, and B, C and D become rank-256 Boolean updates.  A
// closure is unique, so the result is the same 0/1 matrix whatever the band
// width; the wider band cuts the number of full passes over X (each D pass
// reads and writes all n^2 bytes) by 8.
//   * normalize: every nonzero byte becomes 1 (nonzero = edge);
//   * per band [k0, k0 + Bk):
//       diag  -- one workgroup: the block as 256-bit rows in LDS, then the
//                iterative algorithm over k in the block: every row i with
//                bit k set ORs row k into itself, one barrier per k;
//       panels, rest -- gemm_kernel with the 0/1 output (tcu_gemm.hip).
#include "tcu_device.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kBand = 256;           // pivot band width (vertices)
constexpr int kDiagThreads = 1024;   // 16 waves; 2 row words each
constexpr int kWordsPerRow = kBand / 32;

// Every nonzero byte of the n x n matrix becomes 1.  Rows are walked by
// workgroups; with vec (16-byte aligned rows) 16 bytes per thread at a time.
__device__ __forceinline__ unsigned nonzero_bytes(unsigned x) {
  unsigned t = x | (x >> 4);   // low nibble of each byte: OR of its halves
  t |= t >> 2;                 // bits 0, 1: OR of the byte's bit pairs
  t |= t >> 1;                 // bit 0: OR of all 8 bits of the byte
  return t & 0x01010101u;
}

__global__ __launch_bounds__(256) void tc_normalize_kernel(unsigned char *__restrict__ X,
                                                           int64_t n, int64_t ld, int vec) {
  const int64_t full = vec ? n / 16 * 16 : 0;
  for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
    unsigned char *row = X + r * ld;
    for (int64_t c = 16 * (int64_t)threadIdx.x; c < full; c += 16 * (int64_t)blockDim.x) {
      u32x4 v = *(const u32x4 *)(row + c);
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = nonzero_bytes(v[q]);
      *(u32x4 *)(row + c) = v;
    }
    for (int64_t c = full + threadIdx.x; c < n; c += blockDim.x) row[c] = row[c] != 0;
  }
}

// Close the Bk x Bk diagonal block at D (row pitch ld), Bk <= 256.
__global__ __launch_bounds__(kDiagThreads) void tc_diag_kernel(unsigned char *__restrict__ D,
                                                               int64_t ld, int Bk) {
  __shared__ unsigned bits[kBand][kWordsPerRow];
  const int t = threadIdx.x;
  const int i = t >> 2;                  // row
  const int w0 = 2 * (t & 3);            // this thread's two words of row i
  // bytes -> bits (bit b of word w = column 32w + b)
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int w = w0 + q;
    unsigned word = 0;
    if (i < Bk) {
      const unsigned char *row = D + (int64_t)i * ld + 32 * w;
      for (int b = 0; b < 32; ++b)
        if (32 * w + b < Bk && row[b] != 0) word |= 1u << b;
    }
    bits[i][w] = word;
  }
  __syncthreads();
  // The iterative algorithm on the block, k in order.  Bit k of row i is
  // stable during step k (row k only ORs itself into itself), so one
  // barrier per step orders every read and write.
  for (int k = 0; k < Bk; ++k) {
    if ((bits[i][k >> 5] >> (k & 31)) & 1u) {
      bits[i][w0] |= bits[k][w0];
      bits[i][w0 + 1] |= bits[k][w0 + 1];
    }
    __syncthreads();
  }
  // bits -> bytes
  if (i < Bk) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int w = w0 + q;
      const unsigned word = bits[i][w];
      unsigned char *row = D + (int64_t)i * ld + 32 * w;
      for (int b = 0; b < 32; ++b)
        if (32 * w + b < Bk) row[b] = (unsigned char)((word >> b) & 1u);
    }
  }
}

}  // namespace

hipError_t launch_tc(unsigned char *X, int64_t ld, int64_t n, hipStream_t stream, int num_cus) {
  if (n <= 0) return hipSuccess;
  const int64_t rows_grid = n < (int64_t)num_cus * 8 ? n : (int64_t)num_cus * 8;
  const int vec = (ld % 16 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0) ? 1 : 0;
  hipLaunchKernelGGL(tc_normalize_kernel, dim3((unsigned)rows_grid), dim3(256), 0, stream, X, n,
                     ld, vec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int64_t k0 = 0; k0 < n; k0 += kBand) {
    const int Bk = (int)(n - k0 < kBand ? n - k0 : kBand);
    hipLaunchKernelGGL(tc_diag_kernel, dim3(1), dim3(kDiagThreads), 0, stream,
                       X + k0 * ld + k0, ld, Bk);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n == Bk) break;
    e = launch_tc_panels(X, ld, (int)n, (int)k0, Bk, stream);
    if (e != hipSuccess) return e;
    e = launch_tc_rest(X, ld, (int)n, (int)k0, Bk, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace tcu
