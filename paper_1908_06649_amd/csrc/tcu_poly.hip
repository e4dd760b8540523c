// Batch polynomial evaluation of Theorem 11 (Section 4.8):
// out[i] = A(x_i) = sum_{h<n} a_h x_i^h for p points x_i.
//
// The theorem's method, fused into one launch:
//   * X (p x s): row i holds x_i^0 .. x_i^(s-1);
//   * the coefficients, read column-major, form the s x (n/s) matrix with
//     entry (k, j) = a_(k + j s); its s x s blocks are the unit's weights;
//   * C = X times that matrix, as n/m tall calls of p rows (one per block);
//   * A(x_i) = sum_j C[i][j] x_i^(j s).
// Each wave owns chunks of 16 points, one point per matrix-core column:
//   * it computes the powers of its points in binary32 (the theorem's
//     initial exponentiation, as a ladder of squarings shared by all lanes
//     plus a short chain per lane) and hands X to the unit as an unevaluated
//     sum of two bfloat16 words, X = X_hi + X_lo, so the unit multiplies X
//     to about 2^-17 relative accuracy instead of one 16-bit rounding -- the
//     model multiplies exactly, and one rounding of x^k would dominate the
//     error;
//   * for every block it loads the block's weights once (16-byte contiguous
//     runs of coefficients, shared by the wave's U chunks) and issues two
//     matrix-core products per 16-column half (X_hi, then X_lo into the
//     same binary32 accumulators);
//   * binary16 inputs are driven through the unit in bfloat16 too: the
//     5-bit exponent of a binary16 word cannot hold x^k for small |x|
//     (x^(S-1) below 2^-14 loses bits, below 2^-25 vanishes), while bfloat16
//     has binary32's range.  Each binary16 coefficient is split exactly into
//     two bfloat16 words c_hi + c_lo (its 11 significant bits fit in 8 + 8),
//     and every block takes four products, (X_hi + X_lo)(c_hi + c_lo);
//   * lane (r, g) then holds C[point r][columns 16h + 4g + i] of the block
//     and forms t = sum over them of C y^(16h + i), y = x^s, by Horner's
//     rule in y; the blocks are walked last to first and combined by
//     Horner's rule in y^s (acc = acc * y^s + t), and the lane's factor
//     y^(4g) is applied once -- the final combine, never writing C;
//   * the four lanes holding one point add their sums (cross-lane
//     exchange) and one stores A(x_i).
// Coefficients past n and points past p are zero padding.  Results are
// meaningful while |x|^(n-1) and the partial sums stay within binary32
// range (the theorem assumes evaluation without overflow or underflow).
#include "tcu_device.h"
#include "tcu_split.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kPolyThreads = 256;  // 4 waves per workgroup
constexpr int kPolyU = 4;          // 16-point chunks per wave and pass
constexpr int kPolyLongBlocks = 8; // coefficient blocks from which a pass takes 2 kPolyU chunks

template <int DT>
__device__ __forceinline__ float in_to_f32(unsigned bits16) {
  if constexpr (DT == TCU_F16_F32)
    return (float)__builtin_bit_cast(_Float16, (unsigned short)bits16);
  else
    return bf16_to_f32(bits16);
}

// A word of two binary16 coefficients as the exact sum of two words of
// bfloat16 pairs (11 significant bits in 8 + 8).
__device__ __forceinline__ void f16_pair_to_bf16(unsigned w, unsigned &hi, unsigned &lo,
                                                 SplitConsts sc) {
  const float f0 = (float)bitcast<_Float16>((unsigned short)(w & 0xffffu));
  const float f1 = (float)bitcast<_Float16>((unsigned short)(w >> 16));
  split_bf16x2(f0, f1, hi, lo, sc);
}

// b^(step * g) for lane group g = 0..3 from the ladder b^step, b^(2 step):
// two selects and one product (exact when a factor is 1), no branches.
__device__ __forceinline__ float pow_group(int g, float b1, float b2) {
  const float f1 = (g & 1) ? b1 : 1.f;
  const float f2 = (g & 2) ? b2 : 1.f;
  return f1 * f2;
}

template <int DT, int S, int U>
__global__ __launch_bounds__(kPolyThreads) void poly_kernel(const unsigned char *__restrict__ coef,
                                                            int64_t n,
                                                            const unsigned char *__restrict__ pts,
                                                            int64_t np,
                                                            unsigned char *__restrict__ out,
                                                            int64_t nchunks, int64_t nblocks) {
  // Powers a shorter polynomial never uses (k >= n in X, output columns
  // j >= ceil(n/S) in the combine) are replaced by zeros rather than
  // computed, so they cannot overflow where the polynomial itself does not.
  const int64_t ncols = (n + S - 1) / S;
  constexpr int kRun = S == 32 ? 8 : 4;  // contracted elements per lane
  constexpr int kH = S / 16;             // 16-column halves of a block
  typedef typename std::conditional<kRun == 8, u32x4, u32x2>::type Run;
  constexpr int kWords = kRun / 2;
  // The unit runs in bfloat16 for every input type (binary16 coefficients
  // split into two bfloat16 words each, see above).
  constexpr bool kF16 = DT == TCU_F16_F32;
  constexpr int UDT = TCU_BF16_F32;

  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const SplitConsts sc = split_consts();
  // Wave-uniform chunk indices (readfirstlane: the compiler cannot prove
  // threadIdx.x >> 6 uniform), so point addresses are a scalar base plus a
  // per-lane 32-bit offset.
  const int64_t wave = (int64_t)blockIdx.x * (kPolyThreads / 64) +
                       __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * (kPolyThreads / 64);
  const unsigned short *pt16 = (const unsigned short *)pts;
  const unsigned short *cf16 = (const unsigned short *)coef;

  for (int64_t t0 = wave * U; t0 < nchunks; t0 += nwaves * U) {
    Run xh[U], xl[U];
    float yv[U], y16v[U], yg[U], acc[U], ystep[U];
    // All U points first, so their loads are in flight together; points
    // past np read as zero bits (+0 in both formats), and a pass whose
    // points all exist takes no range test.
    const int64_t p0 = t0 * 16;
    const bool whole = p0 + 16 * U <= np;   // every point of the pass exists
    const unsigned short *pp = pt16 + p0;
    unsigned short praw[U];
    if (whole) {
#pragma unroll
      for (int u = 0; u < U; ++u) praw[u] = pp[16 * u + r];
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t idx = p0 + 16 * u + r;
        praw[u] = idx < np ? pt16[idx] : (unsigned short)0;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float x = in_to_f32<DT>(praw[u]);
      // Power ladder (same products in every lane): x^2 .. x^16, y = x^S.
      const float x2 = x * x, x4 = x2 * x2, x8 = x4 * x4, x16 = x8 * x8;
      // X fragment: x^(kRun g + e), e < kRun, as hi + lo words.
      float pw[kRun];
      pw[0] = kRun == 8 ? pow_group(g, x8, x16) : pow_group(g, x4, x8);
#pragma unroll
      for (int e = 1; e < kRun; ++e) pw[e] = pw[e - 1] * x;
      if (n < S) {   // powers past the polynomial's degree are not used
#pragma unroll
        for (int e = 0; e < kRun; ++e) pw[e] = kRun * g + e < n ? pw[e] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < kWords; ++q) {
        unsigned hi, lo;
        split_bf16x2(pw[2 * q], pw[2 * q + 1], hi, lo, sc);
        xh[u][q] = hi;
        xl[u][q] = lo;
      }
      // The combine: column c = 16h + 4g + i of a block has weight
      // y^c = y^(4g) y^(16h) y^i, y = x^S; a lane forms its columns' sum by
      // Horner's rule in y (and y^16 across the halves), the blocks by
      // Horner's rule in y^S, and applies y^(4g) once at the end.  A power
      // that only multiplies unused (zero) columns is replaced by 0, so that
      // it cannot overflow where the polynomial does not: every power kept
      // divides x^(n-1).
      const float y = S == 32 ? x16 * x16 : x16;
      const float y2 = y * y, y4 = y2 * y2, y8 = y4 * y4, y16 = y8 * y8;
      yv[u] = ncols >= 2 ? y : 0.f;
      y16v[u] = ncols > 16 ? y16 : 0.f;
      yg[u] = 4 * g < ncols ? pow_group(g, y4, y8) : 0.f;
      ystep[u] = S == 32 ? y16 * y16 : y16;
      acc[u] = 0.f;
    }

    // Weights of block J: row 16h + r of the unit operand is output column
    // J*S + 16h + r, i.e. the S coefficients starting at (J*S + 16h + r)*S;
    // this lane's run starts kRun*g further.  Blocks wholly inside the
    // coefficient array (a wave-uniform test) take plain vector loads.
    auto load_block = [&](int64_t J, Run (&wb)[kH]) __attribute__((always_inline)) {
      const bool full = (J + 1) * S * S <= n;
      const unsigned short *cb = cf16 + J * S * S;   // wave-uniform block base
#pragma unroll
      for (int h = 0; h < kH; ++h) {
        const int off = (16 * h + r) * S + kRun * g;
        if (full) {
          wb[h] = *(const Run *)(cb + off);
        } else {
          const int64_t left = n - J * S * S - off;
          unsigned ww[kWords];
#pragma unroll
          for (int q = 0; q < kWords; ++q) ww[q] = 0;
#pragma unroll
          for (int e = 0; e < kRun; ++e)
            if (e < left) ww[e >> 1] |= (unsigned)cb[off + e] << (16 * (e & 1));
#pragma unroll
          for (int q = 0; q < kWords; ++q) wb[h][q] = ww[q];
        }
      }
    };
    for (int64_t J = nblocks - 1; J >= 0; --J) {
      Run wf[kH], wl[kH];
      load_block(J, wf);
      if constexpr (kF16) {
#pragma unroll
        for (int h = 0; h < kH; ++h)
#pragma unroll
          for (int q = 0; q < kWords; ++q) {
            unsigned hi, lo;
            f16_pair_to_bf16(wf[h][q], hi, lo, sc);
            wf[h][q] = hi;
            wl[h][q] = lo;
          }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float t = 0.f;
#pragma unroll
        for (int h = 0; h < kH; ++h) {
          f32x4 d;
          if constexpr (S == 32) {
            d = mfma_k32(UDT, wf[h], xh[u], f32x4{0.f, 0.f, 0.f, 0.f});
            d = mfma_k32(UDT, wf[h], xl[u], d);
            if constexpr (kF16) {
              d = mfma_k32(UDT, wl[h], xh[u], d);
              d = mfma_k32(UDT, wl[h], xl[u], d);
            }
          } else {
            d = mfma_k16(UDT, wf[h], xh[u], f32x4{0.f, 0.f, 0.f, 0.f});
            d = mfma_k16(UDT, wf[h], xl[u], d);
            if constexpr (kF16) {
              d = mfma_k16(UDT, wl[h], xh[u], d);
              d = mfma_k16(UDT, wl[h], xl[u], d);
            }
          }
          const float th = __builtin_fmaf(
              __builtin_fmaf(__builtin_fmaf(d[3], yv[u], d[2]), yv[u], d[1]), yv[u], d[0]);
          t = h == 0 ? th : __builtin_fmaf(th, y16v[u], t);
        }
        // Horner over the blocks, last block first: acc = acc * y^S + t.
        acc[u] = J == nblocks - 1 ? t : acc[u] * ystep[u] + t;
      }
    }

#pragma unroll
    for (int u = 0; u < U; ++u) {
      float v = acc[u] * yg[u];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0 && (whole || p0 + 16 * u + r < np)) {
        if constexpr (DT == TCU_BF16_BF16)
          ((unsigned short *)out + p0)[16 * u + r] =
              (unsigned short)(pack_bf16x2(v, 0.f) & 0xffffu);
        else
          ((float *)out + p0)[16 * u + r] = v;
      }
    }
  }
}

template <int DT, int S, int U>
hipError_t launch_poly_u(const void *coef, int64_t n, const void *pts, int64_t np, void *out,
                         hipStream_t stream, int num_cus) {
  const int64_t nchunks = (np + 15) / 16;
  const int64_t nblocks = (n + (int64_t)S * S - 1) / ((int64_t)S * S);
  const int64_t want = (nchunks + 4 * U - 1) / (4 * U);
  const int64_t cap = (int64_t)num_cus * 4;
  const int blocks = (int)(want < cap ? want : cap);
  hipLaunchKernelGGL((poly_kernel<DT, S, U>), dim3(blocks), dim3(kPolyThreads), 0, stream,
                     (const unsigned char *)coef, n, (const unsigned char *)pts, np,
                     (unsigned char *)out, nchunks, nblocks);
  return hipGetLastError();
}

// Each pass of a wave loads every coefficient block once for its U chunks
// of 16 points: long polynomials (8 or more blocks) take 8 chunks per pass,
// halving the coefficient traffic per point.
template <int DT, int S>
hipError_t launch_poly_one(const void *coef, int64_t n, const void *pts, int64_t np, void *out,
                           hipStream_t stream, int num_cus) {
  const int64_t nblocks = (n + (int64_t)S * S - 1) / ((int64_t)S * S);
  if (nblocks >= kPolyLongBlocks)
    return launch_poly_u<DT, S, 2 * kPolyU>(coef, n, pts, np, out, stream, num_cus);
  return launch_poly_u<DT, S, kPolyU>(coef, n, pts, np, out, stream, num_cus);
}

}  // namespace

hipError_t launch_poly(int dtype, int s, const void *coef, int64_t n, const void *pts, int64_t np,
                       void *out, hipStream_t stream, int num_cus) {
  switch (dtype * 2 + (s == 32 ? 1 : 0)) {
    case TCU_F16_F32 * 2 + 0: return launch_poly_one<TCU_F16_F32, 16>(coef, n, pts, np, out, stream, num_cus);
    case TCU_F16_F32 * 2 + 1: return launch_poly_one<TCU_F16_F32, 32>(coef, n, pts, np, out, stream, num_cus);
    case TCU_BF16_F32 * 2 + 0: return launch_poly_one<TCU_BF16_F32, 16>(coef, n, pts, np, out, stream, num_cus);
    case TCU_BF16_F32 * 2 + 1: return launch_poly_one<TCU_BF16_F32, 32>(coef, n, pts, np, out, stream, num_cus);
    case TCU_BF16_BF16 * 2 + 0: return launch_poly_one<TCU_BF16_BF16, 16>(coef, n, pts, np, out, stream, num_cus);
    case TCU_BF16_BF16 * 2 + 1: return launch_poly_one<TCU_BF16_BF16, 32>(coef, n, pts, np, out, stream, num_cus);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcu
