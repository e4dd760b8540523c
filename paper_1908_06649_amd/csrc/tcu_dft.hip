// Discrete Fourier transform by Cooley-Tukey on the tensor unit (Section
// 4.5, Theorem 7): y[k] = sum_j x[j] exp(-2 pi i j k / n), for a batch of
// complex vectors (binary32 real and imaginary parts, interleaved).
//
// The section arranges x as an s x (n/s) matrix, replaces every column by
// its DFT -- the tall product X^T W_s, n/s rows through the unit -- scales
// entry (r, c) by the twiddle w_n^(r c), transposes, and recurses on the s
// rows (a last level of radix n/s^(L-1) <= s).  Here each level -- or two
// consecutive full-radix levels at once (dft_pair_kernel, through LDS) -- is
// one launch that reads the whole array and writes it reordered (a Stockham
// ordering: the digits of k already produced are kept as the fastest-varying
// index), so the last level leaves y in natural order with no separate
// transpose.  With n = R_1 ... R_L, P_t = R_1 ... R_(t-1) and N_t = n / P_t:
//   level t reads  a[j] = src[j (n/R_t) + c],           c = J P_t + K,
//   and writes     dst[(J R_t + k) P_t + K] = w_(N_t)^(J k) sum_j a[j] w_(R_t)^(j k)
// for every transform c < n/R_t (J < N_t/R_t, K < P_t) and k < R_t.
//
// On the unit: 16 transforms per wave, one per matrix-core column; the
// weights operand is W_(R_t) (rows = output frequency k, contracted index j),
// formed once per wave.  Complex products are real products on the bf16
// matrix cores: Re = Wr Xr - Wi Xi, Im = Wi Xr + Wr Xi.  The data and W each
// enter as the sum of two bf16 words (hi + lo), and every real product is
// formed as hi*hi + hi*lo + lo*hi into binary32 accumulators, about 2^-16
// relative accuracy (one bf16 rounding would cost 2^-9 per level).  The
// twiddles are computed in the kernel: for N_t <= 2^20 as the product of two
// entries of per-workgroup LDS tables (each the sincospi of an exact angle),
// above that as one sincospi of the exactly reduced angle; nothing is
// stored between launches.
#include <mutex>

#include "tcu_device.h"
#include "tcu_split.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kDftThreads = 256;

typedef float f32x2 __attribute__((ext_vector_type(2)));

// exp(-2 pi i m / N) for 0 <= m < N, N a power of two: (cos, -sin) of pi x,
// x = 2m/N formed exactly (N is a power of two).
__device__ __forceinline__ f32x2 twiddle(int64_t m, int64_t N) {
  const float x = (float)m * (2.0f / (float)N);
  float s, c;
  sincospif(x, &s, &c);
  return f32x2{c, -s};
}

// Complex product of two (re, im) pairs.
__device__ __forceinline__ f32x2 cmul(f32x2 a, f32x2 b) {
  return f32x2{a[0] * b[0] - a[1] * b[1], a[0] * b[1] + a[1] * b[0]};
}

// Twiddles of one level, N = 2^L: for L <= kTabLg,
//   w_N^m = T_hi[m >> b] * T_lo[m mod 2^b],   b = ceil(L / 2),
// T_lo[i] = w_N^i (i < 2^b) and T_hi[i] = w_N^(i 2^b) (i < 2^(L-b)), built
// in LDS by the workgroup (2^b + 2^(L-b) <= 2048 sincospi evaluations, in
// place of about three per lane and transform step); above kTabLg every
// twiddle is one sincospi.  The choice depends on L alone, so every kernel
// computes the same twiddle bit for bit.
constexpr int kTabLg = 20;
__host__ __device__ constexpr int tab_entries(int L) {
  return L <= kTabLg ? (1 << ((L + 1) / 2)) + (1 << (L / 2)) : 0;
}
struct TwTab {
  const f32x2 *lo = nullptr;   // LDS; null: no table
  const f32x2 *hi = nullptr;
  int b = 0;
  int lg = 0;                  // L
};
// Fill pool[0 .. tab_entries(L)) (threads tid < nthreads share the work);
// the caller synchronises the workgroup before the first lookup.
__device__ __forceinline__ TwTab build_tab(f32x2 *pool, int L, int tid, int nthreads) {
  TwTab t;
  t.lg = L;
  if (L > kTabLg) return t;
  t.b = (L + 1) / 2;
  const int nlo = 1 << t.b, nhi = 1 << (L - t.b);
  const int64_t N = (int64_t)1 << L;
  for (int i = tid; i < nlo + nhi; i += nthreads)
    pool[i] = i < nlo ? twiddle(i, N) : twiddle((int64_t)(i - nlo) << t.b, N);
  t.lo = pool;
  t.hi = pool + nlo;
  return t;
}
// w_N^(m mod N).
__device__ __forceinline__ f32x2 tw(const TwTab &t, int64_t m) {
  const int64_t mm = m & (((int64_t)1 << t.lg) - 1);
  if (t.lo == nullptr) return twiddle(mm, (int64_t)1 << t.lg);
  return cmul(t.hi[mm >> t.b], t.lo[mm & ((1 << t.b) - 1)]);
}

// Shapes of a radix-S step on the unit: a lane holds kRun consecutive
// contracted elements, and the S output frequencies come in kH halves of 16.
template <int S>
struct DftShape {
  static constexpr int kRun = S == 32 ? 8 : 4;   // contracted elements per lane
  static constexpr int kH = S / 16;              // 16-frequency halves
  static constexpr int kWords = kRun / 2;
  typedef typename std::conditional<kRun == 8, u32x4, u32x2>::type Run;
};

// The weights operand W_R (R <= S) as hi/lo words: row k = 16h + r of the
// unit operand, contracted run j = kRun g + e, value w_R^(j k) (zero
// outside R x R); -Wi for the real part.  wtab[m] = w_R^m.
template <int S>
struct DftWeights {
  typedef typename DftShape<S>::Run Run;
  Run wr_h[DftShape<S>::kH], wr_l[DftShape<S>::kH], wi_h[DftShape<S>::kH],
      wi_l[DftShape<S>::kH], ni_h[DftShape<S>::kH], ni_l[DftShape<S>::kH];
};
template <int S>
__device__ __forceinline__ void dft_weights(DftWeights<S> &W, const f32x2 *wtab, int R, int r,
                                            int g, SplitConsts sc) {
  constexpr int kRun = DftShape<S>::kRun, kH = DftShape<S>::kH, kWords = DftShape<S>::kWords;
#pragma unroll
  for (int h = 0; h < kH; ++h) {
    float cr[kRun], ci[kRun];
    const int k = 16 * h + r;
#pragma unroll
    for (int e = 0; e < kRun; ++e) {
      const int j = kRun * g + e;
      const f32x2 w = (j < R && k < R) ? wtab[(j * k) & (R - 1)] : f32x2{0.f, 0.f};
      cr[e] = w[0];
      ci[e] = w[1];
    }
#pragma unroll
    for (int q = 0; q < kWords; ++q) {
      unsigned hi, lo;
      split_bf16x2(cr[2 * q], cr[2 * q + 1], hi, lo, sc);
      W.wr_h[h][q] = hi;
      W.wr_l[h][q] = lo;
      split_bf16x2(ci[2 * q], ci[2 * q + 1], hi, lo, sc);
      W.wi_h[h][q] = hi;
      W.wi_l[h][q] = lo;
      W.ni_h[h][q] = hi ^ 0x80008000u;   // -Wi: flip both signs
      W.ni_l[h][q] = lo ^ 0x80008000u;
    }
  }
}

// One transform column of the unit (lane (r, g) holds its elements
// j = kRun g + e): the data as hi/lo words, then for half h the real and
// imaginary parts of outputs 16h + 4g + i, i < 4 (the matrix-core output
// layout), each real product formed as hi*hi + hi*lo + lo*hi.
template <int S>
struct DftData {
  typename DftShape<S>::Run xr_h, xr_l, xi_h, xi_l;
};
template <int S>
__device__ __forceinline__ void dft_data(DftData<S> &X, const float *xr, const float *xi,
                                         SplitConsts sc) {
#pragma unroll
  for (int q = 0; q < DftShape<S>::kWords; ++q) {
    unsigned hi, lo;
    split_bf16x2(xr[2 * q], xr[2 * q + 1], hi, lo, sc);
    X.xr_h[q] = hi;
    X.xr_l[q] = lo;
    split_bf16x2(xi[2 * q], xi[2 * q + 1], hi, lo, sc);
    X.xi_h[q] = hi;
    X.xi_l[q] = lo;
  }
}
template <int S>
__device__ __forceinline__ void dft_half(const DftWeights<S> &W, const DftData<S> &X, int h,
                                         f32x4 &re, f32x4 &im) {
  typedef typename DftShape<S>::Run Run;
  auto mma = [&](const Run &w, const Run &x, f32x4 d) __attribute__((always_inline)) {
    if constexpr (S == 32)
      return mfma_k32(TCU_BF16_F32, w, x, d);
    else
      return mfma_k16(TCU_BF16_F32, w, x, d);
  };
  re = f32x4{0.f, 0.f, 0.f, 0.f};
  im = f32x4{0.f, 0.f, 0.f, 0.f};
  re = mma(W.wr_h[h], X.xr_h, re);
  re = mma(W.wr_h[h], X.xr_l, re);
  re = mma(W.wr_l[h], X.xr_h, re);
  re = mma(W.ni_h[h], X.xi_h, re);
  re = mma(W.ni_h[h], X.xi_l, re);
  re = mma(W.ni_l[h], X.xi_h, re);
  im = mma(W.wi_h[h], X.xr_h, im);
  im = mma(W.wi_h[h], X.xr_l, im);
  im = mma(W.wi_l[h], X.xr_h, im);
  im = mma(W.wr_h[h], X.xi_h, im);
  im = mma(W.wr_h[h], X.xi_l, im);
  im = mma(W.wr_l[h], X.xi_h, im);
}
// Outputs k0 .. k0+3 of transform J times the twiddles w_(N_t)^(J k):
// w^(J k0), then repeated products with step = w^J.
__device__ __forceinline__ void dft_twiddle4(f32x2 (&y)[4], int64_t J, int k0, const TwTab &tab,
                                             f32x2 step) {
  f32x2 w = tw(tab, J * k0);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    y[i] = cmul(y[i], w);
    if (i < 3) w = cmul(w, step);
  }
}

// One level.  n, R, P, N_t are powers of two and enter as their base-2
// logarithms; ntrans = batch * n / R transforms, 16 per wave step.
template <int S>
__global__ __launch_bounds__(kDftThreads) void dft_level_kernel(
    const f32x2 *__restrict__ src, f32x2 *__restrict__ dst, int lg_n, int lg_r, int lg_p,
    int64_t ntrans) {
  constexpr int kRun = DftShape<S>::kRun, kH = DftShape<S>::kH;
  __shared__ f32x2 wtab[S];               // w_R^m, m < R
  __shared__ f32x2 pool[tab_entries(kTabLg)];

  const int R = 1 << lg_r;
  const int lg_pv = lg_n - lg_r;          // log2 of the transforms per vector
  const int lg_nt = lg_n - lg_p;          // log2 N_t
  const bool last = lg_nt == lg_r;        // N_t = R: no twiddles
  const bool contiguous = lg_p == 0 && R >= 4;   // a lane's 4 outputs are adjacent

  if (threadIdx.x < (unsigned)R) wtab[threadIdx.x] = twiddle(threadIdx.x, R);
  TwTab tab;
  if (!last) tab = build_tab(pool, lg_nt, threadIdx.x, kDftThreads);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const SplitConsts sc = split_consts();
  DftWeights<S> W;
  dft_weights<S>(W, wtab, R, r, g, sc);

  const int64_t wave = (int64_t)blockIdx.x * (kDftThreads / 64) + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * (kDftThreads / 64);
  const int64_t nchunks = (ntrans + 15) >> 4;
  for (int64_t chunk = wave; chunk < nchunks; chunk += nwaves) {
    const int64_t tr = chunk * 16 + r;   // this lane's transform
    const bool live = tr < ntrans;
    const int64_t b = live ? tr >> lg_pv : 0;
    const int64_t c = live ? tr & (((int64_t)1 << lg_pv) - 1) : 0;
    const f32x2 *vin = src + (b << lg_n) + c;
    // data: a[j], j = kRun g + e
    float xr[kRun], xi[kRun];
#pragma unroll
    for (int e = 0; e < kRun; ++e) {
      const int j = kRun * g + e;
      f32x2 v = {0.f, 0.f};
      if (live && j < R) v = vin[(int64_t)j << lg_pv];
      xr[e] = v[0];
      xi[e] = v[1];
    }
    DftData<S> X;
    dft_data<S>(X, xr, xi, sc);
    const int64_t J = c >> lg_p, K = c & (((int64_t)1 << lg_p) - 1);
    f32x2 *vout = dst + (b << lg_n) + ((J << lg_r) << lg_p) + K;
    const f32x2 step = last ? f32x2{1.f, 0.f} : tw(tab, J);
#pragma unroll
    for (int h = 0; h < kH; ++h) {
      f32x4 re, im;
      dft_half<S>(W, X, h, re, im);
      const int k0 = 16 * h + 4 * g;
      if (!live || k0 >= R) continue;
      f32x2 y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) y[i] = f32x2{re[i], im[i]};
      if (!last) dft_twiddle4(y, J, k0, tab, step);
      if (contiguous) {   // outputs k0 .. k0+3 of transform J: 32 adjacent bytes
        f32x4 *o = (f32x4 *)(vout + k0);
        o[0] = f32x4{y[0][0], y[0][1], y[1][0], y[1][1]};
        o[1] = f32x4{y[2][0], y[2][1], y[3][0], y[3][1]};
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (k0 + i < R) vout[(int64_t)(k0 + i) << lg_p] = y[i];
      }
    }
  }
}


// Two consecutive levels t, t+1 of radix S in one launch (both R = S, and
// P_t >= 16 or P_t = 1).  With P = P_t, N' = N_t / S and P' = P S, level
// t+1's transform (J', K' = k P + K) reads output k of level t's
// transforms J = J' + j' (N'/S), j' < S, with the same K.  So the S x S
// values of group (J', K) -- level t's transforms J (rows j') by their
// outputs k -- are formed and consumed inside one workgroup, through LDS:
//   * a workgroup takes 16 groups at once: 16 consecutive K (P >= 16,
//     kLaneK) or 16 consecutive J' (P = 1), so that the level-t loads and
//     the level-(t+1) stores of the 16 matrix-core columns are contiguous;
//   * level t: S steps j' (a wave takes every 4th), each the 16 groups'
//     transforms J = J' + j' (N'/S) as in dft_level_kernel (all of a wave's
//     loads issued first), outputs times w_(N_t)^(J k) into the LDS tile
//     T[group][j'][k];
//   * level t+1: S steps, each 16 transforms over j' read from the tiles
//     (kLaneK: output k of the 16 groups; otherwise 16 consecutive k of one
//     group), outputs times w_(N')^(J' k') unless it is the last level,
//     stored in level t+1's Stockham order.
// Every value takes the same operations as with two dft_level_kernel
// launches (the same weights, products, twiddles, binary32 between the
// levels), so the result is the same bit for bit; only the array's trip
// through HBM between the two levels is saved.
constexpr int kPairGroups = 16;
template <int S>
constexpr int pair_row() { return S + 1; }                          // j' rows, padded
template <int S>
constexpr int pair_group() { return S * pair_row<S>() + 1; }       // one group's tile

constexpr int kPairThreads = 512;   // 8 waves: two per SIMD

template <int S, bool kLaneK>
__global__ __launch_bounds__(kPairThreads) void dft_pair_kernel(
    const f32x2 *__restrict__ src, f32x2 *__restrict__ dst, int lg_n, int lg_p, int64_t ntiles,
    int last2) {
  constexpr int kRun = DftShape<S>::kRun, kH = DftShape<S>::kH;
  constexpr int lg_s = S == 32 ? 5 : 4;
  constexpr int kWaves = kPairThreads / 64;
  constexpr int kSteps = S / kWaves;                // level steps per wave
  constexpr int kRow = pair_row<S>(), kGrp = pair_group<S>();
  __shared__ f32x2 wtab[S];
  __shared__ f32x2 tile[kPairGroups * kGrp];
  // level t's table (N_t <= 2^20) and level t+1's (N' = N_t / S), or one
  // of them: at most 2^10 + 2^10 + 2^(10 - lg_s/2) + 2^(10 - lg_s/2) entries
  constexpr int kPool = tab_entries(kTabLg) + tab_entries(kTabLg - (S == 32 ? 5 : 4));
  __shared__ f32x2 pool[kPool];

  const int lg_nt = lg_n - lg_p;             // level t: N_t
  const int lg_n2 = lg_nt - lg_s;            // level t+1: N' = N_t / S
  const int lg_jp = lg_n2 - lg_s;            // log2 (N'/S): the J' range
  const int lg_pv = lg_n - lg_s;             // n / S: level t's element stride

  if (threadIdx.x < (unsigned)S) wtab[threadIdx.x] = twiddle(threadIdx.x, S);
  const TwTab tab1 = build_tab(pool, lg_nt, threadIdx.x, kPairThreads);
  TwTab tab2;
  if (!last2) tab2 = build_tab(pool + tab_entries(lg_nt), lg_n2, threadIdx.x, kPairThreads);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int wv = threadIdx.x >> 6;
  const SplitConsts sc = split_consts();
  DftWeights<S> W;
  dft_weights<S>(W, wtab, S, r, g, sc);

  // tiles per vector: (N'/S) (P/16) with kLaneK, (N'/S)/16 otherwise
  const int lg_tpv = kLaneK ? lg_jp + lg_p - 4 : lg_jp - 4;
  for (int64_t q = blockIdx.x; q < ntiles; q += gridDim.x) {
    const int64_t b = q >> lg_tpv;
    const int64_t ql = q & (((int64_t)1 << lg_tpv) - 1);
    const f32x2 *vsrc = src + (b << lg_n);
    f32x2 *vdst = dst + (b << lg_n);
    // this lane's group: J'_r and K_r
    const int64_t Jp = kLaneK ? ql >> (lg_p - 4) : (ql << 4) + r;
    const int64_t Kr = kLaneK ? ((ql & (((int64_t)1 << (lg_p - 4)) - 1)) << 4) + r : 0;

    // ---- level t: the wave's steps j' = wv + kWaves i, loads issued first
    f32x2 v[kSteps][kRun];
#pragma unroll
    for (int i = 0; i < kSteps; ++i) {
      const int64_t J = Jp + ((int64_t)(wv + kWaves * i) << lg_jp);
      const f32x2 *vin = vsrc + (J << lg_p) + Kr;
#pragma unroll
      for (int e = 0; e < kRun; ++e) v[i][e] = vin[(int64_t)(kRun * g + e) << lg_pv];
    }
#pragma unroll
    for (int i = 0; i < kSteps; ++i) {
      const int jp = wv + kWaves * i;
      const int64_t J = Jp + ((int64_t)jp << lg_jp);
      float xr[kRun], xi[kRun];
#pragma unroll
      for (int e = 0; e < kRun; ++e) {
        xr[e] = v[i][e][0];
        xi[e] = v[i][e][1];
      }
      DftData<S> X;
      dft_data<S>(X, xr, xi, sc);
      const f32x2 step = tw(tab1, J);
#pragma unroll
      for (int h = 0; h < kH; ++h) {
        f32x4 re, im;
        dft_half<S>(W, X, h, re, im);
        const int k0 = 16 * h + 4 * g;
        f32x2 y[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = f32x2{re[e], im[e]};
        dft_twiddle4(y, J, k0, tab1, step);
        f32x2 *t = tile + r * kGrp + jp * kRow + k0;
#pragma unroll
        for (int e = 0; e < 4; ++e) t[e] = y[e];
      }
    }
    __syncthreads();

    // ---- level t+1: the wave's steps
#pragma unroll
    for (int i = 0; i < kSteps; ++i) {
      const int ch = wv + kWaves * i;
      int grp, k;
      if constexpr (kLaneK) {
        grp = r;
        k = ch;
      } else {
        grp = ch / (S / 16);
        k = 16 * (ch % (S / 16)) + r;
      }
      const int64_t J2 = kLaneK ? Jp : (ql << 4) + grp;          // level t+1's J'
      const int64_t K2 = ((int64_t)k << lg_p) + (kLaneK ? Kr : 0);
      float xr[kRun], xi[kRun];
      const f32x2 *t = tile + grp * kGrp + k;
#pragma unroll
      for (int e = 0; e < kRun; ++e) {
        const f32x2 a = t[(kRun * g + e) * kRow];
        xr[e] = a[0];
        xi[e] = a[1];
      }
      DftData<S> X;
      dft_data<S>(X, xr, xi, sc);
      f32x2 *vout = vdst + ((J2 << lg_s) << (lg_p + lg_s)) + K2;
      const f32x2 step = last2 ? f32x2{1.f, 0.f} : tw(tab2, J2);
#pragma unroll
      for (int h = 0; h < kH; ++h) {
        f32x4 re, im;
        dft_half<S>(W, X, h, re, im);
        const int k0 = 16 * h + 4 * g;
        f32x2 y[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = f32x2{re[e], im[e]};
        if (!last2) dft_twiddle4(y, J2, k0, tab2, step);
#pragma unroll
        for (int e = 0; e < 4; ++e) vout[(int64_t)(k0 + e) << (lg_p + lg_s)] = y[e];
      }
    }
    __syncthreads();   // the tiles are rewritten by the next iteration
  }
}

// Scratch of the allocation-free DFT (tcu_dft_noalloc): the levels' second
// buffer.  In host code this name is only a stand-in for the symbol; the
// array's device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[TCU_DFT_NOALLOC_MAX_BYTES];

int ilog2(int64_t v) {
  int l = 0;
  while (((int64_t)1 << l) < v) ++l;
  return l;
}

// Whether levels t, t+1 (radix S each, P = P_t) run as one pair launch:
// both full radix, and a coalesced lane order exists (16 consecutive K, or
// P = 1 with at least 16 groups J' per vector).
bool pair_ok(int64_t n, int s, int64_t P) {
  const int64_t n2 = n / P / s;   // N' = N_t / s
  if (n2 < s) return false;       // level t+1 would not have full radix
  if (knob(TCU_KNOB_DFT_PAIRS) == 1) return false;   // test override: single levels
  return P >= 16 || (P == 1 && n2 / s >= 16);
}

template <int S>
hipError_t launch_pair(const f32x2 *src, f32x2 *dst, int64_t n, int64_t P, int64_t batch,
                       bool last2, hipStream_t stream, int num_cus) {
  const int64_t ntiles = batch * (n / ((int64_t)S * S)) / kPairGroups;
  const int64_t cap = num_cus;      // one workgroup per CU (the tiles take most of the LDS)
  const int blocks = (int)(ntiles < cap ? ntiles : cap);
  if (P >= 16)
    hipLaunchKernelGGL((dft_pair_kernel<S, true>), dim3(blocks), dim3(kPairThreads), 0, stream,
                       src, dst, ilog2(n), ilog2(P), ntiles, last2 ? 1 : 0);
  else
    hipLaunchKernelGGL((dft_pair_kernel<S, false>), dim3(blocks), dim3(kPairThreads), 0, stream,
                       src, dst, ilog2(n), ilog2(P), ntiles, last2 ? 1 : 0);
  return hipGetLastError();
}

template <int S>
hipError_t launch_level(const f32x2 *src, f32x2 *dst, int64_t n, int R, int64_t P,
                        int64_t batch, hipStream_t stream, int num_cus) {
  const int64_t ntrans = batch * (n / R);
  const int64_t nchunks = (ntrans + 15) / 16;
  const int64_t want = (nchunks + 3) / 4;
  const int64_t cap = (int64_t)num_cus * 8;
  const int blocks = (int)(want < cap ? want : cap);
  hipLaunchKernelGGL((dft_level_kernel<S>), dim3(blocks), dim3(kDftThreads), 0, stream, src, dst,
                     ilog2(n), ilog2(R), ilog2(P), ntrans);
  return hipGetLastError();
}

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxScratchDevices] = {};

// The scratch array's address on the current device (each device holds its
// own copy), resolved with that device current on its first use there.
hipError_t scratch_on_current_device(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

int dft_levels(int64_t n, int s) {
  int L = 1;
  for (int64_t m = s; m < n; m *= s) ++L;
  return L;
}

hipError_t launch_dft(const void *x, void *y, void *work, int64_t n, int64_t batch, int s,
                      hipStream_t stream, int num_cus) {
  if (n <= 0 || batch <= 0) return hipSuccess;
  const int L = dft_levels(n, s);
  // Launches: levels taken two at a time where pair_ok holds, else one
  // (decided once, before anything is launched).
  bool pairs[64];
  int launches = 0;
  {
    int64_t P = 1;
    for (int t = 1; t <= L;) {
      const bool pair = t < L && pair_ok(n, s, P);
      P *= pair ? (int64_t)s * s : (t < L ? s : n / P);
      t += pair ? 2 : 1;
      pairs[launches++] = pair;
    }
  }
  int64_t P = 1;
  const f32x2 *src = (const f32x2 *)x;
  int launch = 0;
  for (int t = 1; t <= L;) {
    const bool pair = pairs[launch];
    // the launches alternate between work and y so that the last lands in y
    ++launch;
    f32x2 *dst = (f32x2 *)(((launches - launch) % 2 == 0) ? y : work);
    hipError_t e;
    if (pair) {
      const bool last2 = t + 1 == L;
      e = s == 32 ? launch_pair<32>(src, dst, n, P, batch, last2, stream, num_cus)
                  : launch_pair<16>(src, dst, n, P, batch, last2, stream, num_cus);
      P *= (int64_t)s * s;
      t += 2;
    } else {
      const int R = (int)(t < L ? s : n / P);
      e = s == 32 ? launch_level<32>(src, dst, n, R, P, batch, stream, num_cus)
                  : launch_level<16>(src, dst, n, R, P, batch, stream, num_cus);
      P *= R;
      t += 1;
    }
    if (e != hipSuccess) return e;
    src = dst;
  }
  return hipSuccess;
}

hipError_t launch_dft_noalloc(const void *x, void *y, int64_t n, int64_t batch, int s,
                              hipStream_t stream, int num_cus) {
  if (n <= 0 || batch <= 0) return hipSuccess;
  void *work = nullptr;
  if (dft_levels(n, s) > 1) {
    const hipError_t e = scratch_on_current_device(&work);
    if (e != hipSuccess) return e;
  }
  return launch_dft(x, y, work, n, batch, s, stream, num_cus);
}

}  // namespace tcu
