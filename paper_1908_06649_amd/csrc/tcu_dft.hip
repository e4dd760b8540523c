// Discrete Fourier transform by Cooley-Tukey on the tensor unit (Section
// 4.5, Theorem 7): y[k] = sum_j x[j] exp(-2 pi i j k / n), for a batch of
// complex vectors (binary32 real and imaginary parts, interleaved).
//
// The section arranges x as an s x (n/s) matrix, replaces every column by
// its DFT -- the tall product X^T W_s, n/s rows through the unit -- scales
// entry (r, c) by the twiddle w_n^(r c), transposes, and recurses on the s
// rows (a last level of radix n/s^(L-1) <= s).  Here each level is one
// launch that reads the whole array and writes it reordered (a Stockham
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
// twiddles are computed in the kernel (sincospi of an exactly reduced
// angle); nothing is precomputed or stored.
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

// One level.  n, R, P, N_t are powers of two and enter as their base-2
// logarithms; ntrans = batch * n / R transforms, 16 per wave step.
template <int S>
__global__ __launch_bounds__(kDftThreads) void dft_level_kernel(
    const f32x2 *__restrict__ src, f32x2 *__restrict__ dst, int lg_n, int lg_r, int lg_p,
    int64_t ntrans) {
  constexpr int kRun = S == 32 ? 8 : 4;   // contracted elements per lane
  constexpr int kH = S / 16;              // 16-frequency halves
  constexpr int kWords = kRun / 2;
  typedef typename std::conditional<kRun == 8, u32x4, u32x2>::type Run;
  __shared__ f32x2 wtab[S];               // w_R^m, m < R

  const int R = 1 << lg_r;
  const int lg_pv = lg_n - lg_r;          // log2 of the transforms per vector
  const int lg_nt = lg_n - lg_p;          // log2 N_t
  const int64_t nt_mask = ((int64_t)1 << lg_nt) - 1;
  const bool last = lg_nt == lg_r;        // N_t = R: no twiddles
  const bool contiguous = lg_p == 0 && R >= 4;   // a lane's 4 outputs are adjacent

  if (threadIdx.x < (unsigned)R) wtab[threadIdx.x] = twiddle(threadIdx.x, R);
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const SplitConsts sc = split_consts();

  // Weights operand: row k = 16h + r, contracted run j = kRun g + e, value
  // w_R^(j k) (zero outside R x R), as hi/lo words; -Wi for the real part.
  Run wr_h[kH], wr_l[kH], wi_h[kH], wi_l[kH], ni_h[kH], ni_l[kH];
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
      wr_h[h][q] = hi;
      wr_l[h][q] = lo;
      split_bf16x2(ci[2 * q], ci[2 * q + 1], hi, lo, sc);
      wi_h[h][q] = hi;
      wi_l[h][q] = lo;
      ni_h[h][q] = hi ^ 0x80008000u;   // -Wi: flip both signs
      ni_l[h][q] = lo ^ 0x80008000u;
    }
  }

  const int64_t wave = (int64_t)blockIdx.x * (kDftThreads / 64) + (threadIdx.x >> 6);
  const int64_t nwaves = (int64_t)gridDim.x * (kDftThreads / 64);
  const int64_t nchunks = (ntrans + 15) >> 4;
  for (int64_t chunk = wave; chunk < nchunks; chunk += nwaves) {
    const int64_t tr = chunk * 16 + r;   // this lane's transform
    const bool live = tr < ntrans;
    const int64_t b = live ? tr >> lg_pv : 0;
    const int64_t c = live ? tr & (((int64_t)1 << lg_pv) - 1) : 0;
    const f32x2 *vin = src + (b << lg_n) + c;
    // data: a[j], j = kRun g + e, as hi/lo words of the real and imaginary parts
    float xr[kRun], xi[kRun];
#pragma unroll
    for (int e = 0; e < kRun; ++e) {
      const int j = kRun * g + e;
      f32x2 v = {0.f, 0.f};
      if (live && j < R) v = vin[(int64_t)j << lg_pv];
      xr[e] = v[0];
      xi[e] = v[1];
    }
    Run xr_h, xr_l, xi_h, xi_l;
#pragma unroll
    for (int q = 0; q < kWords; ++q) {
      unsigned hi, lo;
      split_bf16x2(xr[2 * q], xr[2 * q + 1], hi, lo, sc);
      xr_h[q] = hi;
      xr_l[q] = lo;
      split_bf16x2(xi[2 * q], xi[2 * q + 1], hi, lo, sc);
      xi_h[q] = hi;
      xi_l[q] = lo;
    }
    const int64_t J = c >> lg_p, K = c & (((int64_t)1 << lg_p) - 1);
    f32x2 *vout = dst + (b << lg_n) + ((J << lg_r) << lg_p) + K;
    // twiddle w_(N_t)^(J k) for k = k0 + i: w^(J k0) times step^i, step = w^J
    const f32x2 step = last ? f32x2{1.f, 0.f} : twiddle(J & nt_mask, (int64_t)1 << lg_nt);
#pragma unroll
    for (int h = 0; h < kH; ++h) {
      f32x4 re = {0.f, 0.f, 0.f, 0.f}, im = {0.f, 0.f, 0.f, 0.f};
      auto mma = [&](const Run &w, const Run &x, f32x4 d) __attribute__((always_inline)) {
        if constexpr (S == 32)
          return mfma_k32(TCU_BF16_F32, w, x, d);
        else
          return mfma_k16(TCU_BF16_F32, w, x, d);
      };
      re = mma(wr_h[h], xr_h, re);
      re = mma(wr_h[h], xr_l, re);
      re = mma(wr_l[h], xr_h, re);
      re = mma(ni_h[h], xi_h, re);
      re = mma(ni_h[h], xi_l, re);
      re = mma(ni_l[h], xi_h, re);
      im = mma(wi_h[h], xr_h, im);
      im = mma(wi_h[h], xr_l, im);
      im = mma(wi_l[h], xr_h, im);
      im = mma(wr_h[h], xi_h, im);
      im = mma(wr_h[h], xi_l, im);
      im = mma(wr_l[h], xi_h, im);
      const int k0 = 16 * h + 4 * g;
      if (!live || k0 >= R) continue;
      f32x2 y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) y[i] = f32x2{re[i], im[i]};
      if (!last) {
        f32x2 w = twiddle((J * k0) & nt_mask, (int64_t)1 << lg_nt);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          y[i] = cmul(y[i], w);
          if (i < 3) w = cmul(w, step);
        }
      }
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

// Scratch of the allocation-free DFT (tcu_dft_noalloc): the levels' second
// buffer.  In host code this name is only a stand-in for the symbol; the
// array's device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[TCU_DFT_NOALLOC_MAX_BYTES];

int ilog2(int64_t v) {
  int l = 0;
  while (((int64_t)1 << l) < v) ++l;
  return l;
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
  int64_t P = 1;
  const f32x2 *src = (const f32x2 *)x;
  for (int t = 1; t <= L; ++t) {
    const int R = (int)(t < L ? s : n / P);
    // the levels alternate between work and y so that the last lands in y
    f32x2 *dst = (f32x2 *)(((L - t) % 2 == 0) ? y : work);
    const hipError_t e = s == 32 ? launch_level<32>(src, dst, n, R, P, batch, stream, num_cus)
                                 : launch_level<16>(src, dst, n, R, P, batch, stream, num_cus);
    if (e != hipSuccess) return e;
    src = dst;
    P *= R;
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
