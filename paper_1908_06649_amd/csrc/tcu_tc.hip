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
//                of 32 (see tc_diag_kernel);
//       panels, rest -- the product kernels with the 0/1 output: the
//                pivot column band, then the pivot row band and the rest
//                in one launch (tcu_gemm.hip explains why the in-place
//                updates may overlap).
#include "tcu_device.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kBand = 256;           // pivot band width (vertices)
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

// 4 bytes holding 0/1 -> 4 bits, and back.
__device__ __forceinline__ unsigned bytes_to_bits4(unsigned x) {
  return (x & 1u) | ((x >> 7) & 2u) | ((x >> 14) & 4u) | ((x >> 21) & 8u);
}
__device__ __forceinline__ unsigned bits4_to_bytes(unsigned b) {
  return (b & 1u) | ((b & 2u) << 7) | ((b & 4u) << 14) | ((b & 8u) << 21);
}

// Value of lane h (0..3) of each group of 4 consecutive lanes (DPP quad
// permutation; h wave-uniform).
__device__ __forceinline__ unsigned quad_broadcast(unsigned v, int h) {
  switch (h) {
    case 0: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x00, 0xf, 0xf, false);
    case 1: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x55, 0xf, 0xf, false);
    case 2: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xaa, 0xf, 0xf, false);
    default: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xff, 0xf, 0xf, false);
  }
}

// Close the Bk x Bk diagonal block at D (row pitch ld; entries already 0/1),
// Bk <= 256.  Row i is held as 8 words of bits by the 4 threads 4i .. 4i+3
// (two words each).  The pivots are taken in sub-bands K of 32; for each:
//   * the pivots' current rows are published to LDS;
//   * one wave closes the 32 x 32 block of K's rows and columns (the
//     iterative algorithm on 32 one-word rows, the pivot row broadcast with
//     readlane), giving T*[k]: the pivots reachable from pivot k through K,
//     k included;
//   * every row i (pivot or not) forms R_i, the union of T*[k] over the
//     pivots k it has an edge to, and ORs in the published rows of R_i.
// That is the iterative algorithm's 32 steps over K: a vertex reaches v
// through K exactly when some pivot it reaches through K has an edge to v.
// Both unions over a 32-bit set are taken 4 bits at a time from tables of
// all 16 unions of 4 consecutive pivots' words (8 lookups instead of 32
// masked terms): tab1 over T*, tab2 over each word of the published rows.
// A wave's lookups into tab2 touch the regions of 4 words at once; regions
// kTab2Pitch = 136 words apart start 8 banks further on per word, so the
// four regions (even words) fall on disjoint 16-bank windows and a lookup
// is conflict-free (16 subsets of one region lie in 16 distinct banks).
template <bool kVec>
__global__ __launch_bounds__(1024) void tc_diag_kernel(unsigned char *__restrict__ D, int64_t ld,
                                                       int Bk) {
  __shared__ __attribute__((aligned(16))) unsigned krow[32][kWordsPerRow];
  __shared__ unsigned tab1[8 * 16];                  // [group][subset]
  constexpr int kTab2Pitch = 8 * 16 + 8;
  __shared__ unsigned tab2[kWordsPerRow * kTab2Pitch];   // [word][group][subset]
  const int t = threadIdx.x;
  const int i = t >> 2;              // row
  const int w0 = 2 * (t & 3);        // this thread's words w0, w0 + 1 of row i
  unsigned row[2];
  // bytes -> bits (bit b of word w = column 32w + b)
  const unsigned char *src = D + (int64_t)i * ld;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int w = w0 + q;
    unsigned word = 0;
    if (i < Bk) {
      if (kVec && 32 * w + 32 <= Bk) {
        const u32x4 a = *(const u32x4 *)(src + 32 * w);
        const u32x4 b = *(const u32x4 *)(src + 32 * w + 16);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          word |= bytes_to_bits4(a[c]) << (4 * c);
          word |= bytes_to_bits4(b[c]) << (16 + 4 * c);
        }
      } else {
        for (int b = 0; b < 32; ++b)
          if (32 * w + b < Bk && src[32 * w + b]) word |= 1u << b;
      }
    }
    row[q] = word;
  }
#pragma unroll
  for (int sb = 0; sb < kWordsPerRow; ++sb) {
    if (32 * sb >= Bk) break;
    const int nk = Bk - 32 * sb < 32 ? Bk - 32 * sb : 32;   // pivots in this sub-band
    const unsigned kmask = nk == 32 ? ~0u : (1u << nk) - 1u;
    if (i >= 32 * sb && i < 32 * sb + 32) {
      krow[i - 32 * sb][w0] = row[0];
      krow[i - 32 * sb][w0 + 1] = row[1];
    }
    __syncthreads();
    // (Pivots past nk have zero rows and no bits in kmask: they add nothing.)
    if (t < 64) {
      // wave 0: lanes 0..31 close the pivot block; then tab1 from T*.
      unsigned tk = t < 32 ? krow[t][sb] & kmask : 0u;
#pragma unroll
      for (int kk = 0; kk < 32; ++kk) {
        const unsigned pivot = (unsigned)__builtin_amdgcn_readlane((int)tk, kk);
        tk |= pivot & (0u - ((tk >> kk) & 1u));
      }
      const unsigned tstar = t < 32 ? (tk | (1u << t)) : 0u;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = t + 64 * h, grp = e >> 4, m = e & 15;
        unsigned v = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const unsigned x = (unsigned)__shfl((int)tstar, 4 * grp + b, 64);
          v |= x & (0u - ((unsigned)(m >> b) & 1u));
        }
        tab1[e] = v;
      }
    }
    {
      // tab2[w][grp][m] = union of word w of the published rows 4 grp + b, b in m
      const int w = t >> 7, grp = (t >> 4) & 7, m = t & 15;
      unsigned v = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) v |= krow[4 * grp + b][w] & (0u - ((unsigned)(m >> b) & 1u));
      tab2[w * kTab2Pitch + (t & 127)] = v;
    }
    __syncthreads();
    // word sb of row i, from the quad lane that holds it
    const unsigned wsb = quad_broadcast((sb & 1) ? row[1] : row[0], sb >> 1);
    const unsigned edges = wsb & kmask;
    unsigned reach = 0;
#pragma unroll
    for (int grp = 0; grp < 8; ++grp) reach |= tab1[16 * grp + ((edges >> (4 * grp)) & 15u)];
    reach &= kmask;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const unsigned *t2 = tab2 + kTab2Pitch * (w0 + q);
      unsigned add = 0;
#pragma unroll
      for (int grp = 0; grp < 8; ++grp) add |= t2[16 * grp + ((reach >> (4 * grp)) & 15u)];
      row[q] |= add;
    }
    __syncthreads();   // krow and the tables are rewritten by the next sub-band
  }
  // bits -> bytes
  if (i < Bk) {
    unsigned char *dst = D + (int64_t)i * ld;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int w = w0 + q;
      if (kVec && 32 * w + 32 <= Bk) {
        u32x4 a, b;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          a[c] = bits4_to_bytes(row[q] >> (4 * c));
          b[c] = bits4_to_bytes(row[q] >> (16 + 4 * c));
        }
        *(u32x4 *)(dst + 32 * w) = a;
        *(u32x4 *)(dst + 32 * w + 16) = b;
      } else {
        for (int b = 0; b < 32; ++b)
          if (32 * w + b < Bk) dst[32 * w + b] = (unsigned char)((row[q] >> b) & 1u);
      }
    }
  }
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
  for (int64_t k0 = 0; k0 < n; k0 += kBand) {
    const int Bk = (int)(n - k0 < kBand ? n - k0 : kBand);
    TCU_TRY(launch_diag(X, ld, k0, Bk, vec, stream));
    if (n == Bk) break;
    TCU_TRY(launch_tc_panels(X, ld, (int)n, (int)k0, Bk, stream));
    TCU_TRY(launch_tc_rest(X, ld, (int)n, (int)k0, Bk, stream, num_cus));
  }
  return hipSuccess;
}

}  // namespace tcu
