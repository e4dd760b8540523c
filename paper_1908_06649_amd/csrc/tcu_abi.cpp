// C ABI of the tensor-unit library: argument validation, unit
// configuration, cost accounting and dispatch to the HIP launchers.
// Every argument check runs before the first HIP call of an entry point.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include <initializer_list>
#include <utility>

#include "tcu.h"
#include "tcu_launch.h"

#define TCU_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// Machine parameters of the model (Section 3): unit size s = sqrt(m), plus
// the element types and the stream the unit is driven on.  Per host thread.
struct UnitConfig {
  int s = 16;
  int dtype = TCU_F16_F32;
  void *stream = nullptr;
};
thread_local UnitConfig g_cfg;

// Test overrides and the pointer-check switch (tcu_set_knob).  Pointer
// checks start on when TCU_DEBUG holds a nonzero integer at load time; the
// environment is read only here, once.
constexpr int kKnobs = 6;
int initial_knob(int k) {
  if (k != TCU_KNOB_CHECK_POINTERS) return 0;
  const char *v = std::getenv("TCU_DEBUG");
  return v && std::atoi(v) != 0 ? 1 : 0;
}
std::atomic<int> g_knob[kKnobs] = {{0}, {0}, {0}, {0}, {initial_knob(TCU_KNOB_CHECK_POINTERS)}, {0}};

std::atomic<int64_t> g_calls{0};
std::atomic<int64_t> g_square_calls{0};
std::atomic<int64_t> g_work{0};

constexpr int kMaxDevices = 64;
struct DeviceInfo {
  int state = 0;  // 0: not probed, 1: usable gfx950, <0: tcu_status
  int num_cus = 0;
};
std::mutex g_dev_mu;
DeviceInfo g_dev[kMaxDevices];
std::atomic<bool> g_runtime_ok{false};

bool unit_ok(int s) { return s == 16 || s == 32; }
bool dtype_ok(int dt) { return dt >= TCU_F16_F32 && dt <= TCU_I8_I32; }
int64_t in_size(int dt) { return dt == TCU_I8_I32 ? 1 : 2; }
int64_t out_size(int dt) { return dt == TCU_BF16_BF16 ? 2 : 4; }
bool misaligned(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }
bool overlap(const void *a, int64_t na, const void *b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// Resolve the current device and check it is a gfx950; fills its CU count.
int device_ready(int *num_cus) {
  if (!g_runtime_ok.load(std::memory_order_acquire)) {
    int count = 0;
    const hipError_t e = hipGetDeviceCount(&count);
    if (e == hipErrorNoDevice || (e == hipSuccess && count <= 0)) return TCU_ERR_NO_DEVICE;
    if (e != hipSuccess) return TCU_ERR_HIP;
    g_runtime_ok.store(true, std::memory_order_release);
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return TCU_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return TCU_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_dev_mu);
  DeviceInfo &d = g_dev[dev];
  if (d.state == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return TCU_ERR_HIP;
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
      d.state = TCU_ERR_UNSUPPORTED;
    } else {
      d.state = 1;
      d.num_cus = prop.multiProcessorCount;
    }
  }
  if (d.state < 0) return d.state;
  *num_cus = d.num_cus;
  return TCU_OK;
}

// Whether [p, p + bytes) lies inside one device allocation of the current
// device (tcu_check_device_range).  A failed query's error is cleared from
// HIP's last-error state unless that state already held an error.
int device_range(const void *p, int64_t bytes) {
  if (bytes < 0) return TCU_ERR_SHAPE;
  if (bytes == 0) return TCU_OK;
  if (!p) return TCU_ERR_POINTER;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return TCU_ERR_HIP;
  const hipError_t before = hipPeekAtLastError();
  auto fail = [&](int status) {
    if (before == hipSuccess) (void)hipGetLastError();
    return status;
  };
  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof(attr));
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) return fail(TCU_ERR_POINTER);
  if ((attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) ||
      attr.device != dev)
    return TCU_ERR_POINTER;
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, const_cast<void *>(p)) != hipSuccess)
    return fail(TCU_ERR_POINTER);
  const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
  if (q < b || q - b > size || (uint64_t)bytes > size - (q - b)) return TCU_ERR_POINTER;
  return TCU_OK;
}

// With pointer checks on, every operand extent (pointer, bytes) in turn.
int check_ranges(std::initializer_list<std::pair<const void *, int64_t>> ranges) {
  if (g_knob[TCU_KNOB_CHECK_POINTERS].load(std::memory_order_relaxed) == 0) return TCU_OK;
  for (const auto &r : ranges) {
    const int rc = device_range(r.first, r.second);
    if (rc != TCU_OK) return rc;
  }
  return TCU_OK;
}

int validate_tall(const void *A, int64_t n, int s, const void *B, const void *C, int dt) {
  if (!A || !B || !C) return TCU_ERR_NULL;
  if (!unit_ok(s) || !dtype_ok(dt)) return TCU_ERR_UNSUPPORTED;
  // The model requires n >= sqrt(m) rows for a call (Section 3).
  if (n < s || n > TCU_MAX_ROWS) return TCU_ERR_SHAPE;
  if (misaligned(A) || misaligned(B) || misaligned(C)) return TCU_ERR_ALIGN;
  const int64_t a_bytes = n * s * in_size(dt);
  const int64_t b_bytes = (int64_t)s * s * in_size(dt);
  const int64_t c_bytes = n * s * out_size(dt);
  if (overlap(C, c_bytes, A, a_bytes) || overlap(C, c_bytes, B, b_bytes)) return TCU_ERR_OVERLAP;
  return TCU_OK;
}

int validate_gemm(const void *A, const void *B, const void *C, int64_t N, int s, int dt) {
  if (!A || !B || !C) return TCU_ERR_NULL;
  if (!unit_ok(s) || !dtype_ok(dt)) return TCU_ERR_UNSUPPORTED;
  // Theorem 2 takes N a multiple of s (the strips and blocks tile A and B).
  if (N < s || N % s != 0 || N > TCU_MAX_ORDER) return TCU_ERR_SHAPE;
  // int32 sums of N products of magnitude <= 2^14 stay exact while N < 2^17.
  if (dt == TCU_I8_I32 && N >= ((int64_t)1 << 17)) return TCU_ERR_SHAPE;
  if (misaligned(A) || misaligned(B) || misaligned(C)) return TCU_ERR_ALIGN;
  const int64_t in_bytes = N * N * in_size(dt);
  const int64_t c_bytes = N * N * out_size(dt);
  if (overlap(C, c_bytes, A, in_bytes) || overlap(C, c_bytes, B, in_bytes)) return TCU_ERR_OVERLAP;
  return TCU_OK;
}

// Bytes from the base of an R x C view with row pitch ld (elements of es
// bytes) to one past its last element; 0 for an empty view.  Formed in
// 128-bit arithmetic and saturated at 2^62, so that no combination of
// in-range arguments (R up to 2^30 rows of pitch up to 2^62) can wrap
// around and pass a size check.
int64_t view_extent(int64_t rows, int64_t cols, int64_t ld, int64_t es) {
  if (rows <= 0 || cols <= 0) return 0;
  const __int128 e = ((__int128)(rows - 1) * ld + cols) * es;
  constexpr int64_t kSat = (int64_t)1 << 62;
  return e > (__int128)kSat ? kSat : (int64_t)e;
}

// Whether two row-major views (base, rows, bytes per row, byte pitch) share
// a byte.  Disjoint address ranges never do.  Views with one byte pitch P
// (a single-row view takes the other's pitch) are laid on one grid of
// P-byte rows and tested as rectangles, so disjoint blocks of one array
// (the D functions of Sections 4.2 and 4.3 work on such blocks) pass.
// Other overlapping ranges are reported as overlapping.
bool views_overlap(const void *a, int64_t ar, int64_t aw, int64_t ap, const void *b, int64_t br,
                   int64_t bw, int64_t bp) {
  if (ar == 0 || aw == 0 || br == 0 || bw == 0) return false;
  if (!overlap(a, (ar - 1) * ap + aw, b, (br - 1) * bp + bw)) return false;
  if (ar == 1 && br == 1) return true;
  if (ar == 1 && aw <= bp) ap = bp;
  if (br == 1 && bw <= ap) bp = ap;
  if (ap != bp) return true;
  const int64_t P = ap;
  const int64_t d = (int64_t)(reinterpret_cast<uintptr_t>(b) - reinterpret_cast<uintptr_t>(a));
  int64_t q = d / P, c = d % P;
  if (c < 0) {
    c += P;
    q -= 1;
  }
  // In a's grid, row i of b covers bytes [c, c + bw) of grid row q + i,
  // continuing into grid row q + i + 1 when c + bw > P.
  auto hits = [&](int64_t r0, int64_t c0, int64_t c1) {
    return r0 < ar && r0 + br > 0 && c0 < aw && c1 > 0;
  };
  if (hits(q, c, c + bw < P ? c + bw : P)) return true;
  return c + bw > P && hits(q + 1, 0, c + bw - P);
}

int validate_rect(const void *A, int64_t lda, const void *B, int64_t ldb, const void *C,
                  int64_t ldc, int64_t M, int64_t K, int64_t N, int flags, int s, int dt) {
  if (!unit_ok(s) || !dtype_ok(dt) || (flags & ~TCU_ACCUMULATE) != 0) return TCU_ERR_UNSUPPORTED;
  if (M < 0 || K < 0 || N < 0 || M > TCU_MAX_RECT_DIM || K > TCU_MAX_RECT_DIM ||
      N > TCU_MAX_RECT_DIM)
    return TCU_ERR_SHAPE;
  // A pointer may be NULL only if its matrix has no elements.
  if ((!A && M * K > 0) || (!B && K * N > 0) || (!C && M * N > 0)) return TCU_ERR_NULL;
  // int32 sums of K products of magnitude <= 2^14 stay exact while K < 2^17.
  if (dt == TCU_I8_I32 && K >= ((int64_t)1 << 17)) return TCU_ERR_SHAPE;
  constexpr int64_t kMaxExtent = (int64_t)1 << 40;
  if (lda < K || ldb < N || ldc < N || lda >= kMaxExtent || ldb >= kMaxExtent ||
      ldc >= kMaxExtent)
    return TCU_ERR_SHAPE;
  const int64_t ea = view_extent(M, K, lda, in_size(dt));
  const int64_t eb = view_extent(K, N, ldb, in_size(dt));
  const int64_t ec = view_extent(M, N, ldc, out_size(dt));
  if (ea >= kMaxExtent || eb >= kMaxExtent || ec >= kMaxExtent) return TCU_ERR_SHAPE;
  if (misaligned(A) || misaligned(B) || misaligned(C)) return TCU_ERR_ALIGN;
  const int64_t ci = in_size(dt), co = out_size(dt);
  if (views_overlap(C, M, N * co, ldc * co, A, M, K * ci, lda * ci) ||
      views_overlap(C, M, N * co, ldc * co, B, K, N * ci, ldb * ci))
    return TCU_ERR_OVERLAP;
  return TCU_OK;
}

int validate_poly(const void *coef, int64_t n, const void *pts, int64_t p, const void *out, int s,
                  int dt) {
  if (!unit_ok(s) || !dtype_ok(dt) || dt == TCU_I8_I32) return TCU_ERR_UNSUPPORTED;
  if (n < 0 || p < 0 || n > TCU_MAX_ROWS || p > TCU_MAX_ROWS) return TCU_ERR_SHAPE;
  // A pointer may be NULL only if its array is empty.
  if ((!coef && n > 0) || (!pts && p > 0) || (!out && p > 0)) return TCU_ERR_NULL;
  if (misaligned(coef) || misaligned(pts) || misaligned(out)) return TCU_ERR_ALIGN;
  const int64_t ob = p * out_size(dt);
  if (overlap(out, ob, coef, n * 2) || overlap(out, ob, pts, p * 2)) return TCU_ERR_OVERLAP;
  return TCU_OK;
}

int validate_tc(const void *X, int64_t n, int64_t ld, int s) {
  if (!unit_ok(s)) return TCU_ERR_UNSUPPORTED;
  if (n < 0 || n > TCU_MAX_RECT_DIM || ld < n) return TCU_ERR_SHAPE;
  if (!X && n > 0) return TCU_ERR_NULL;
  if (n > 0 && view_extent(n, n, ld, 1) >= ((int64_t)1 << 40)) return TCU_ERR_SHAPE;
  if (misaligned(X)) return TCU_ERR_ALIGN;
  return TCU_OK;
}

// The DFT's checks other than its work buffer: unit size, n, batch,
// extent, x and y (null, alignment, overlap).  *need_work: whether the
// transform has more than one level (its levels then need a second buffer).
int validate_dft_xy(const void *x, const void *y, int64_t n, int64_t batch, int s,
                    bool *need_work) {
  if (!unit_ok(s)) return TCU_ERR_UNSUPPORTED;
  if (n < 1 || n > TCU_MAX_DFT_N || (n & (n - 1)) != 0 || batch < 0) return TCU_ERR_SHAPE;
  // batch * n * 8 bytes must stay below 2^40
  if (batch > 0 && n > (((int64_t)1 << 40) - 1) / 8 / batch) return TCU_ERR_SHAPE;
  const int64_t bytes = batch * n * 8;
  *need_work = tcu::dft_levels(n, s) > 1;
  if (bytes > 0 && (!x || !y)) return TCU_ERR_NULL;
  if (misaligned(x) || misaligned(y)) return TCU_ERR_ALIGN;
  if (overlap(y, bytes, x, bytes)) return TCU_ERR_OVERLAP;
  return TCU_OK;
}

int validate_dft(const void *x, const void *y, const void *work, int64_t n, int64_t batch, int s) {
  bool need_work = false;
  const int rc = validate_dft_xy(x, y, n, batch, s, &need_work);
  if (rc != TCU_OK) return rc;
  const int64_t bytes = batch * n * 8;
  if (bytes > 0 && need_work && !work) return TCU_ERR_NULL;
  if (misaligned(work)) return TCU_ERR_ALIGN;
  if (need_work && (overlap(work, bytes, x, bytes) || overlap(work, bytes, y, bytes)))
    return TCU_ERR_OVERLAP;
  return TCU_OK;
}

// Theorem 7's cost accounting of one transform of `batch` vectors.
void count_dft(int64_t n, int64_t batch, int s) {
  const int L = tcu::dft_levels(n, s);
  int64_t P = 1, calls = 0, squares = 0;
  for (int t = 1; t <= L; ++t) {
    const int64_t R = t < L ? s : n / P;
    const int64_t rows = n / R;
    calls += 4 * batch;
    squares += 4 * batch * ((rows + s - 1) / s);
    P *= R;
  }
  g_calls.fetch_add(calls, std::memory_order_relaxed);
  g_square_calls.fetch_add(squares, std::memory_order_relaxed);
  g_work.fetch_add(squares * s * s, std::memory_order_relaxed);
}

}  // namespace

TCU_EXPORT int tcu_set_unit(int s) {
  if (!unit_ok(s)) return TCU_ERR_UNSUPPORTED;
  g_cfg.s = s;
  return TCU_OK;
}
TCU_EXPORT int tcu_get_unit(void) { return g_cfg.s; }

TCU_EXPORT int tcu_set_dtype(int dtype) {
  if (!dtype_ok(dtype)) return TCU_ERR_UNSUPPORTED;
  g_cfg.dtype = dtype;
  return TCU_OK;
}
TCU_EXPORT int tcu_get_dtype(void) { return g_cfg.dtype; }

TCU_EXPORT int tcu_set_stream(void *hip_stream) {
  g_cfg.stream = hip_stream;
  return TCU_OK;
}
TCU_EXPORT void *tcu_get_stream(void) { return g_cfg.stream; }

TCU_EXPORT int tcu_mm_tall_ex(const void *A, int64_t n, int s, const void *B, void *C, int dtype,
                              void *hip_stream) {
  int rc = validate_tall(A, n, s, B, C, dtype);
  if (rc != TCU_OK) return rc;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  rc = check_ranges({{A, n * s * in_size(dtype)}, {B, (int64_t)s * s * in_size(dtype)},
                     {C, n * s * out_size(dtype)}});
  if (rc != TCU_OK) return rc;
  if (tcu::launch_tall(dtype, s, A, n, B, C, false, (hipStream_t)hip_stream, num_cus) !=
      hipSuccess)
    return TCU_ERR_HIP;
  g_calls.fetch_add(1, std::memory_order_relaxed);
  g_square_calls.fetch_add((n + s - 1) / s, std::memory_order_relaxed);
  g_work.fetch_add(n * s, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_mm_tall(const void *A, int64_t n, int s, const void *B, void *C) {
  if (!A || !B || !C) return TCU_ERR_NULL;
  if (s != g_cfg.s) return TCU_ERR_UNSUPPORTED;
  return tcu_mm_tall_ex(A, n, s, B, C, g_cfg.dtype, g_cfg.stream);
}

TCU_EXPORT int tcu_gemm_ex(const void *A, const void *B, void *C, int64_t N, int s, int dtype,
                           void *hip_stream) {
  int rc = validate_gemm(A, B, C, N, s, dtype);
  if (rc != TCU_OK) return rc;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  rc = check_ranges({{A, N * N * in_size(dtype)}, {B, N * N * in_size(dtype)},
                     {C, N * N * out_size(dtype)}});
  if (rc != TCU_OK) return rc;
  const tcu::RectArgs args{A, N, B, N, C, N, N, N, N, false};
  if (tcu::launch_rect(dtype, s, args, (hipStream_t)hip_stream, num_cus) != hipSuccess)
    return TCU_ERR_HIP;
  // Theorem 2: (N/s)^2 calls, each on an N x s strip (N/s weak-model square
  // calls and N*s model work apiece).
  const int64_t q = N / s;
  g_calls.fetch_add(q * q, std::memory_order_relaxed);
  g_square_calls.fetch_add(q * q * q, std::memory_order_relaxed);
  g_work.fetch_add(q * q * N * s, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_gemm(const void *A, const void *B, void *C, int64_t N) {
  return tcu_gemm_ex(A, B, C, N, g_cfg.s, g_cfg.dtype, g_cfg.stream);
}

TCU_EXPORT int tcu_gemm_rect_ex(const void *A, int64_t lda, const void *B, int64_t ldb, void *C,
                                int64_t ldc, int64_t M, int64_t K, int64_t N, int flags, int s,
                                int dtype, void *hip_stream) {
  int rc = validate_rect(A, lda, B, ldb, C, ldc, M, K, N, flags, s, dtype);
  if (rc != TCU_OK) return rc;
  const bool accum = (flags & TCU_ACCUMULATE) != 0;
  // Nothing to store, or C + (empty sum) = C.
  if (M == 0 || N == 0 || (K == 0 && accum)) return TCU_OK;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  rc = check_ranges({{A, view_extent(M, K, lda, in_size(dtype))},
                     {B, view_extent(K, N, ldb, in_size(dtype))},
                     {C, view_extent(M, N, ldc, out_size(dtype))}});
  if (rc != TCU_OK) return rc;
  const tcu::RectArgs args{A, lda, B, ldb, C, ldc, M, K, N, accum};
  if (tcu::launch_rect(dtype, s, args, (hipStream_t)hip_stream, num_cus) != hipSuccess)
    return TCU_ERR_HIP;
  // Corollary 1 via Theorem 2 on the zero-padded operands: ceil(K/s) strips
  // times ceil(N/s) blocks per strip, one call each, every call on all
  // ceil(M/s)*s padded rows.
  const int64_t calls = ((K + s - 1) / s) * ((N + s - 1) / s);
  const int64_t row_blocks = (M + s - 1) / s;
  g_calls.fetch_add(calls, std::memory_order_relaxed);
  g_square_calls.fetch_add(calls * row_blocks, std::memory_order_relaxed);
  g_work.fetch_add(calls * row_blocks * s * s, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_gemm_rect(const void *A, int64_t lda, const void *B, int64_t ldb, void *C,
                             int64_t ldc, int64_t M, int64_t K, int64_t N, int flags) {
  return tcu_gemm_rect_ex(A, lda, B, ldb, C, ldc, M, K, N, flags, g_cfg.s, g_cfg.dtype,
                          g_cfg.stream);
}

TCU_EXPORT int tcu_poly_eval_ex(const void *coef, int64_t n, const void *points, int64_t p,
                                void *out, int s, int dtype, void *hip_stream) {
  int rc = validate_poly(coef, n, points, p, out, s, dtype);
  if (rc != TCU_OK) return rc;
  if (p == 0) return TCU_OK;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  rc = check_ranges({{coef, n * 2}, {points, p * 2}, {out, p * out_size(dtype)}});
  if (rc != TCU_OK) return rc;
  if (tcu::launch_poly(dtype, s, coef, n, points, p, out, (hipStream_t)hip_stream, num_cus) !=
      hipSuccess)
    return TCU_ERR_HIP;
  // Theorem 11: ceil(n/m) calls of X (p x s) times an s x s coefficient
  // block, each issued twice (X as the sum of two bfloat16 words), and
  // twice more for binary16 coefficients (each the sum of two bfloat16
  // words).
  const int64_t per_block = dtype == TCU_F16_F32 ? 4 : 2;
  const int64_t calls = per_block * ((n + (int64_t)s * s - 1) / ((int64_t)s * s));
  const int64_t row_blocks = (p + s - 1) / s;
  g_calls.fetch_add(calls, std::memory_order_relaxed);
  g_square_calls.fetch_add(calls * row_blocks, std::memory_order_relaxed);
  g_work.fetch_add(calls * row_blocks * s * s, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_poly_eval(const void *coef, int64_t n, const void *points, int64_t p,
                             void *out) {
  return tcu_poly_eval_ex(coef, n, points, p, out, g_cfg.s, g_cfg.dtype, g_cfg.stream);
}

TCU_EXPORT int tcu_transitive_closure_ex(void *X, int64_t n, int64_t ld, int s,
                                         void *hip_stream) {
  int rc = validate_tc(X, n, ld, s);
  if (rc != TCU_OK) return rc;
  if (n == 0) return TCU_OK;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  rc = check_ranges({{X, view_extent(n, n, ld, 1)}});
  if (rc != TCU_OK) return rc;
  if (tcu::launch_tc((unsigned char *)X, ld, n, (hipStream_t)hip_stream, num_cus) != hipSuccess)
    return TCU_ERR_HIP;
  // The section's blocked algorithm with s-wide blocks: for each of the
  // q = ceil(n/s) pivots, q - 1 tall calls of the D function (pivot row
  // block X_kj as the weights, the (q - 1) s rows of the other X_ik
  // streamed through).
  const int64_t q = (n + s - 1) / s;
  const int64_t calls = q * (q - 1);
  g_calls.fetch_add(calls, std::memory_order_relaxed);
  g_square_calls.fetch_add(calls * (q - 1), std::memory_order_relaxed);
  g_work.fetch_add(calls * (q - 1) * s * s, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_transitive_closure(void *X, int64_t n, int64_t ld) {
  return tcu_transitive_closure_ex(X, n, ld, g_cfg.s, g_cfg.stream);
}

TCU_EXPORT int tcu_dft_ex(const void *x, void *y, void *work, int64_t n, int64_t batch, int s,
                          void *hip_stream) {
  int rc = validate_dft(x, y, work, n, batch, s);
  if (rc != TCU_OK) return rc;
  if (batch == 0) return TCU_OK;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  const int64_t bytes = batch * n * 8;
  rc = check_ranges({{x, bytes}, {y, bytes}, {work, tcu::dft_levels(n, s) > 1 ? bytes : 0}});
  if (rc != TCU_OK) return rc;
  if (tcu::launch_dft(x, y, work, n, batch, s, (hipStream_t)hip_stream, num_cus) != hipSuccess)
    return TCU_ERR_HIP;
  count_dft(n, batch, s);
  return TCU_OK;
}

TCU_EXPORT int tcu_dft(const void *x, void *y, void *work, int64_t n, int64_t batch) {
  return tcu_dft_ex(x, y, work, n, batch, g_cfg.s, g_cfg.stream);
}

TCU_EXPORT int tcu_dft_noalloc(const void *x, void *y, int64_t n, int64_t batch, int s,
                               void *hip_stream) {
  bool need_work = false;
  int rc = validate_dft_xy(x, y, n, batch, s, &need_work);
  if (rc != TCU_OK) return rc;
  // the levels' second buffer is the library's fixed scratch array
  if (need_work && batch * n * 8 > TCU_DFT_NOALLOC_MAX_BYTES) return TCU_ERR_SCRATCH;
  if (batch == 0) return TCU_OK;
  int num_cus = 0;
  rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  const int64_t bytes = batch * n * 8;
  rc = check_ranges({{x, bytes}, {y, bytes}});
  if (rc != TCU_OK) return rc;
  if (tcu::launch_dft_noalloc(x, y, n, batch, s, (hipStream_t)hip_stream, num_cus) !=
      hipSuccess)
    return TCU_ERR_HIP;
  count_dft(n, batch, s);
  return TCU_OK;
}


TCU_EXPORT int64_t tcu_calls(void) { return g_calls.load(std::memory_order_relaxed); }
TCU_EXPORT int64_t tcu_square_calls(void) { return g_square_calls.load(std::memory_order_relaxed); }
TCU_EXPORT int64_t tcu_work(void) { return g_work.load(std::memory_order_relaxed); }
TCU_EXPORT void tcu_reset_calls(void) {
  g_calls.store(0);
  g_square_calls.store(0);
  g_work.store(0);
}

TCU_EXPORT int tcu_check_device_range(const void *p, int64_t bytes) {
  if (bytes < 0) return TCU_ERR_SHAPE;
  if (bytes == 0) return TCU_OK;
  int num_cus = 0;
  const int rc = device_ready(&num_cus);
  if (rc != TCU_OK) return rc;
  return device_range(p, bytes);
}

TCU_EXPORT int tcu_set_knob(int knob, int value) {
  if (knob < 0 || knob >= kKnobs || value < 0) return TCU_ERR_UNSUPPORTED;
  if (knob == TCU_KNOB_GEMM_KERNEL && value > TCU_PATH_RING) return TCU_ERR_UNSUPPORTED;
  if ((knob == TCU_KNOB_CHECK_POINTERS || knob == TCU_KNOB_DFT_PAIRS) && value > 1)
    return TCU_ERR_UNSUPPORTED;
  g_knob[knob].store(value, std::memory_order_relaxed);
  return TCU_OK;
}

TCU_EXPORT int tcu_get_knob(int knob) {
  if (knob < 0 || knob >= kKnobs) return -1;
  return g_knob[knob].load(std::memory_order_relaxed);
}

namespace tcu {
int knob(int which) {
  return which >= 0 && which < kKnobs ? g_knob[which].load(std::memory_order_relaxed) : 0;
}
}  // namespace tcu

TCU_EXPORT const char *tcu_strerror(int status) {
  switch (status) {
    case TCU_OK: return "success";
    case TCU_ERR_NULL: return "a required pointer is NULL";
    case TCU_ERR_SHAPE: return "invalid shape (n < s, N < s, N not a multiple of s, or too large)";
    case TCU_ERR_UNSUPPORTED: return "unsupported unit size, dtype, or device (gfx950 required)";
    case TCU_ERR_ALIGN: return "a base pointer is not 16-byte aligned";
    case TCU_ERR_OVERLAP: return "the output overlaps an input";
    case TCU_ERR_HIP: return "HIP runtime error";
    case TCU_ERR_NO_DEVICE: return "no HIP device visible";
    case TCU_ERR_POINTER: return "an operand is not inside one device allocation of the current device";
    case TCU_ERR_SCRATCH:
      return "the problem exceeds the fixed scratch of the allocation-free entry point";
  }
  return "unknown tcu status";
}
