// Internal launchers behind the C ABI (host side).  Arguments are already
// validated by the ABI layer; these only pick a kernel instance and launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tcu.h"

namespace tcu {

constexpr int kNoBand = 0x7fffffff;

// Current value of a test override (a TCU_KNOB_* value of tcu.h), set
// through tcu_set_knob; 0 = the automatic choice.
int knob(int which);

// Placement of a full-tile kernel's tile grid in the output: tile row tm
// starts at m_base + 256 tm, plus skip_m once tm >= band_m (the same for
// columns).  The identity by default; the transitive closure uses it to
// step over the pivot bands another launch owns.
struct TileRemap {
  int m_base = 0, band_m = kNoBand, skip_m = 0;
  int n_base = 0, band_n = kNoBand, skip_n = 0;
};

// Native call: C (n x s) = A (n x s) * B (s x s) [+ C when accum], for s in
// {16, 32}, contiguous operands.
hipError_t launch_tall(int dtype, int s, const void *A, int64_t n, const void *B, void *C,
                       bool accum, hipStream_t stream, int num_cus);

// C (M x N) = A (M x K) * B (K x N) [+ C when accum] with row pitches in
// elements; 0 <= M, K, N <= 2^30, M and N positive.  Theorem 2's strips and
// blocks fused into one launch (the square product is M = K = N).
struct RectArgs {
  const void *A;
  int64_t lda;
  const void *B;
  int64_t ldb;
  void *C;
  int64_t ldc;
  int64_t M, K, N;
  bool accum;
};
hipError_t launch_rect(int dtype, int s, const RectArgs &args, hipStream_t stream, int num_cus);

// Transitive closure, in place on an n x n int8 0/1 matrix X with row pitch
// ld: all pivot bands of Bk <= 256 vertices in order (see tcu_tc.hip).
hipError_t launch_tc(unsigned char *X, int64_t ld, int64_t n, hipStream_t stream, int num_cus);
// Its matrix-core phases for the band [k0, k0 + Bk): the pivot column band,
// then the pivot row band together with the rest of the matrix
// (tcu_gemm.hip).
hipError_t launch_tc_panels(unsigned char *X, int64_t ld, int n, int k0, int Bk,
                            hipStream_t stream);
// close_next: the band's D update also closes the next band's diagonal
// block [k0 + Bk, k0 + 2 Bk)^2 (whole 256-wide bands on the full-tile
// kernel only).
hipError_t launch_tc_rest(unsigned char *X, int64_t ld, int n, int k0, int Bk,
                          hipStream_t stream, int num_cus, bool close_next);
// Whether the full-tile kernel takes the D updates (n a multiple of 256,
// whole bands, 16-byte row pitch), and its launch on a remapped tile grid.
bool tc_full_tiles(int64_t n, int Bk, int64_t ld);
// diag_pid >= 0: the tile (in the kernel's tile order) that is the next
// band's diagonal block, closed after its update; -1: none.
hipError_t launch_tc_tiles(unsigned char *X, int64_t ld, int n, int k0, int tiles_m,
                           int tiles_n, const TileRemap &remap, hipStream_t stream,
                           int num_cus, int diag_pid = -1);

// Forward DFT of `batch` complex64 vectors of length n (a power of two):
// ceil(log_s n) Cooley-Tukey levels alternating between work and y, the last
// writing y (see tcu_dft.hip).
int dft_levels(int64_t n, int s);
hipError_t launch_dft(const void *x, void *y, void *work, int64_t n, int64_t batch, int s,
                      hipStream_t stream, int num_cus);
// The same with the levels' second buffer in the library's fixed device
// array (TCU_DFT_NOALLOC_MAX_BYTES; the caller has checked the size); its
// address on the current device is resolved once per device.
hipError_t launch_dft_noalloc(const void *x, void *y, int64_t n, int64_t batch, int s,
                              hipStream_t stream, int num_cus);

// Batch polynomial evaluation: out[i] = sum_{h<n} coef[h] * pts[i]^h for
// i < np, 16-bit inputs (dtype TCU_F16_F32, TCU_BF16_F32 or TCU_BF16_BF16).
hipError_t launch_poly(int dtype, int s, const void *coef, int64_t n, const void *pts, int64_t np,
                       void *out, hipStream_t stream, int num_cus);

}  // namespace tcu
