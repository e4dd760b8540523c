// C ABI of the tensor-unit library: argument validation, unit
// configuration, cost accounting and dispatch to the HIP launchers.
// Every argument check runs before the first HIP call of an entry point.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstring>
#include <mutex>

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
  if (tcu::launch_tall(dtype, s, A, n, B, C, (hipStream_t)hip_stream, num_cus) != hipSuccess)
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
  if (tcu::launch_gemm(dtype, A, B, C, N, (hipStream_t)hip_stream, num_cus) != hipSuccess)
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

TCU_EXPORT int64_t tcu_calls(void) { return g_calls.load(std::memory_order_relaxed); }
TCU_EXPORT int64_t tcu_square_calls(void) { return g_square_calls.load(std::memory_order_relaxed); }
TCU_EXPORT int64_t tcu_work(void) { return g_work.load(std::memory_order_relaxed); }
TCU_EXPORT void tcu_reset_calls(void) {
  g_calls.store(0);
  g_square_calls.store(0);
  g_work.store(0);
}

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
  }
  return "unknown tcu status";
}
