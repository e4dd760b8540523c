// Timing loop for the benchmark's fit of the model's per-call cost
// (Section 3: a call on n rows costs O(n sqrt(m) + l)).  It issues native
// calls back to back from C, so the per-call cost it measures holds no
// Python argument marshalling.  Host code only; built into its own
// library (libtcu_timing.so) next to libtcu.so, which it calls through the
// C ABI like any other client.
#include <hip/hip_runtime.h>

#include <chrono>
#include <cstdint>

#include "tcu.h"

extern "C" __attribute__((visibility("default"))) int tcu_timing_tall_loop(
    const void *A, int64_t n, int s, const void *B, void *C, int dtype, void *stream, int reps,
    double *async_s_per_call, double *sync_s_per_call) {
  // async: reps calls issued back to back, one synchronisation at the end
  // (the steady-state cost of a call in a sequence of calls, as Theorem 2
  // issues them); sync: each call followed by a stream synchronisation (the
  // round trip of a single call).  Both in seconds per call.
  if (reps < 1 || !async_s_per_call || !sync_s_per_call) return TCU_ERR_SHAPE;
  const hipStream_t st = (hipStream_t)stream;
  int rc = tcu_mm_tall_ex(A, n, s, B, C, dtype, stream);
  if (rc != TCU_OK) return rc;
  if (hipStreamSynchronize(st) != hipSuccess) return TCU_ERR_HIP;
  using clk = std::chrono::steady_clock;
  auto t0 = clk::now();
  for (int i = 0; i < reps; ++i) {
    rc = tcu_mm_tall_ex(A, n, s, B, C, dtype, stream);
    if (rc != TCU_OK) return rc;
  }
  if (hipStreamSynchronize(st) != hipSuccess) return TCU_ERR_HIP;
  auto t1 = clk::now();
  *async_s_per_call = std::chrono::duration<double>(t1 - t0).count() / reps;
  const int sync_reps = reps < 200 ? reps : 200;
  t0 = clk::now();
  for (int i = 0; i < sync_reps; ++i) {
    rc = tcu_mm_tall_ex(A, n, s, B, C, dtype, stream);
    if (rc != TCU_OK) return rc;
    if (hipStreamSynchronize(st) != hipSuccess) return TCU_ERR_HIP;
  }
  t1 = clk::now();
  *sync_s_per_call = std::chrono::duration<double>(t1 - t0).count() / sync_reps;
  return TCU_OK;
}
