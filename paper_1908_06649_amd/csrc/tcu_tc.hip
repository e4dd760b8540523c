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
//       diag  -- one workgroup: the block as 256-bit rows in registers, the
//                iterative algorithm over the block's pivots by sub-bands
//                of 32 (close_diag_block in tcu_tc_diag.h); a launch of its
//                own for the first band and, with whole 256-wide bands,
//                done for every later band by one workgroup of the previous
//                band's rest launch, right after it updated the block;
//       panels, rest -- the product kernels with the 0/1 output: the
//                pivot column band, then the pivot row band and the rest
//                in one launch (tcu_gemm.hip explains why the in-place
//                updates may overlap).
#include "tcu_device.h"
#include "tcu_launch.h"
#include "tcu_tc_diag.h"

namespace tcu {
namespace {

constexpr int kBand = kDiagBand;     // pivot band width (vertices)

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

// Close the Bk x Bk diagonal block at D (close_diag_block in tcu_tc_diag.h),
// one workgroup of 1024 threads: row i as 8 words of bits in 4 threads'
// registers.
template <bool kVec>
__global__ __launch_bounds__(1024) void tc_diag_kernel(unsigned char *__restrict__ D, int64_t ld,
                                                       int Bk) {
  __shared__ __attribute__((aligned(16))) DiagShared s;
  close_diag_block<kVec, 1024>(D, ld, Bk, s);
}

hipError_t launch_diag(unsigned char *X, int64_t ld, int64_t k0, int Bk, bool vec,
                       hipStream_t stream) {
  if (vec)
    hipLaunchKernelGGL(tc_diag_kernel<true>, dim3(1), dim3(1024), 0, stream, X + k0 * ld + k0, ld,
                       Bk);
  else
    hipLaunchKernelGGL(tc_diag_kernel<false>, dim3(1), dim3(1024), 0, stream, X + k0 * ld + k0,
                       ld, Bk);
  return hipGetLastError();
}

#define TCU_TRY(x)                   \
  do {                               \
    const hipError_t e_ = (x);       \
    if (e_ != hipSuccess) return e_; \
  } while (0)

}  // namespace

hipError_t launch_tc(unsigned char *X, int64_t ld, int64_t n, hipStream_t stream, int num_cus) {
  if (n <= 0) return hipSuccess;
  const int64_t rows_grid = n < (int64_t)num_cus * 8 ? n : (int64_t)num_cus * 8;
  const bool vec = ld % 16 == 0 && (reinterpret_cast<uintptr_t>(X) & 15) == 0;
  hipLaunchKernelGGL(tc_normalize_kernel, dim3((unsigned)rows_grid), dim3(256), 0, stream, X, n,
                     ld, vec ? 1 : 0);
  TCU_TRY(hipGetLastError());
  // With whole 256-wide bands the D update of band k0 also closes the next
  // band's diagonal block (one workgroup, right after updating that block,
  // while the others update the rest), so only the first band's closure is
  // a launch of its own.
  // Workgroups of the persistent D-update launch: one per CU, or the test
  // override TCU_KNOB_PP_GRID (a tiny grid gives every workgroup many tiles).
  const int pp_grid = knob(TCU_KNOB_PP_GRID) > 0 ? knob(TCU_KNOB_PP_GRID) : num_cus;
  bool diag_closed = false;
  for (int64_t k0 = 0; k0 < n; k0 += kBand) {
    const int Bk = (int)(n - k0 < kBand ? n - k0 : kBand);
    if (!diag_closed) TCU_TRY(launch_diag(X, ld, k0, Bk, vec, stream));
    if (n == Bk) break;
    TCU_TRY(launch_tc_panels(X, ld, (int)n, (int)k0, Bk, stream));
    // (the fused closure needs a second workgroup for the other tiles)
    const bool close_next = vec && pp_grid >= 2 && tc_full_tiles(n, Bk, ld) && k0 + kBand < n &&
                            tc_full_tiles(n, (int)(n - k0 - kBand < kBand ? n - k0 - kBand : kBand), ld);
    TCU_TRY(launch_tc_rest(X, ld, (int)n, (int)k0, Bk, stream, pp_grid, close_next));
    diag_closed = close_next;
  }
  return hipSuccess;
}

}  // namespace tcu
