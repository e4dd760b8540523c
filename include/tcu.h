/*
 * tcu.h -- C ABI of the MI355X (gfx950) tensor-unit library.
 *
 * The library implements the hot path of the (m,l)-TCU model of
 * "A Computational Model for Tensor Core Units" (Chowdhury, Silvestri,
 * Vella):
 *
 *   - tcu_mm_tall: the model's native tensor-unit call, which multiplies an
 *     n x sqrt(m) matrix A by a sqrt(m) x sqrt(m) matrix B in one
 *     instruction naming the addresses of A, B and C and the row count n
 *     (Section 3, definition of the (m,l)-TCU model; the tall left operand is
 *     the model's third property, "asymmetric behavior").
 *   - tcu_gemm: the dense N x N multiplication of Theorem 2 (Section 4.1),
 *     built from (N/s)^2 such calls: A is cut into N x s vertical strips A_i,
 *     B into s x s blocks B_{i,j}, and output strip j is sum_i A_i * B_{i,j}.
 *
 * Throughout, s = sqrt(m) is the unit size (a machine parameter of the
 * model), n is the row count of a tall call and N the order of the square
 * product.
 *
 * Conventions shared by every entry point:
 *   - All matrix pointers are DEVICE pointers (memory of the current HIP
 *     device).  Matrices are row-major and contiguous: element (r, c) of an
 *     R x C matrix is at index r*C + c.
 *   - The caller allocates and frees A, B and C.  The library never
 *     allocates, frees or retains them, and keeps no pointer across calls.
 *   - C is overwritten with the product (the unit stores its result; it does
 *     not accumulate into C).
 *   - Calls are asynchronous on the stream in effect; the caller synchronises.
 *   - Every call returns a tcu_status: 0 on success, a negative code on
 *     failure.  Argument checks (null, shape, unit size, dtype, alignment,
 *     overlap) all run before any HIP call, so a rejected call touches no
 *     device state.  A rejected call leaves C unmodified and does not count
 *     as a tensor-unit call.
 *   - Base pointers must be 16-byte aligned.  C must not overlap A or B
 *     (A and B may overlap each other; both are only read).
 *   - Unit configuration (tcu_set_unit, tcu_set_dtype, tcu_set_stream) is
 *     per host thread.  The call counters are process-wide and atomic.
 */
#ifndef TCU_H
#define TCU_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum tcu_status {
    TCU_OK = 0,
    TCU_ERR_NULL = -1,        /* a required pointer is NULL */
    TCU_ERR_SHAPE = -2,       /* n < s, N < s, N % s != 0, size overflow, ... */
    TCU_ERR_UNSUPPORTED = -3, /* unit size or dtype not supported, or not a gfx950 device */
    TCU_ERR_ALIGN = -4,       /* a base pointer is not 16-byte aligned */
    TCU_ERR_OVERLAP = -5,     /* C overlaps A or B */
    TCU_ERR_HIP = -6,         /* the HIP runtime reported an error (launch, device query) */
    TCU_ERR_NO_DEVICE = -7    /* no HIP device is visible */
} tcu_status;

/* Element types (input, output) of the unit.  Floating-point inputs are
 * multiplied exactly and summed in binary32; int8 inputs are summed exactly
 * in int32 (exact for K <= 2^17 since |a*b| <= 2^14). */
typedef enum tcu_dtype {
    TCU_F16_F32 = 0,    /* binary16 in, binary32 out */
    TCU_BF16_F32 = 1,   /* bfloat16 in, binary32 out */
    TCU_BF16_BF16 = 2,  /* bfloat16 in, bfloat16 out (binary32 sum rounded to nearest even) */
    TCU_I8_I32 = 3      /* int8 in, int32 out */
} tcu_dtype;

/* Largest supported n (tall call) and N (square product). */
#define TCU_MAX_ROWS ((int64_t)1 << 40)
#define TCU_MAX_ORDER ((int64_t)1 << 20)

/* ---- unit configuration (machine parameters of the model, Section 3) ---- */

/* Set the unit size s = sqrt(m) used by tcu_gemm and expected by
 * tcu_mm_tall.  Supported: 16 and 32.  Default 16.
 * Returns TCU_OK or TCU_ERR_UNSUPPORTED (configuration unchanged). */
int tcu_set_unit(int s);
int tcu_get_unit(void);

/* Set the (input, output) element types (a tcu_dtype value).  Default
 * TCU_F16_F32.  Returns TCU_OK or TCU_ERR_UNSUPPORTED. */
int tcu_set_dtype(int dtype);
int tcu_get_dtype(void);

/* Set the hipStream_t that calls are issued on; NULL is the default stream.
 * Always returns TCU_OK.  The stream must belong to the current device. */
int tcu_set_stream(void *hip_stream);
void *tcu_get_stream(void);

/* ---- the native call (Section 3, model definition) ----
 *
 * C (n x s) = A (n x s) * B (s x s).
 *   A: device pointer, n*s input elements, row-major.
 *   n: rows of A and C; the model requires n >= s.  n need not be a multiple
 *      of s (row tails are handled).
 *   s: the unit size; must equal tcu_get_unit() (the machine has one unit).
 *   B: device pointer, s*s input elements, row-major: the "weights" loaded
 *      into the unit once per call.
 *   C: device pointer, n*s output elements, row-major, overwritten.
 * Element types come from tcu_get_dtype(); the stream from tcu_get_stream().
 * Errors: TCU_ERR_NULL, TCU_ERR_SHAPE (n < s, n > TCU_MAX_ROWS),
 * TCU_ERR_UNSUPPORTED (s not the unit size), TCU_ERR_ALIGN, TCU_ERR_OVERLAP,
 * TCU_ERR_NO_DEVICE, TCU_ERR_HIP.
 * On success the logical call counter advances by 1. */
int tcu_mm_tall(const void *A, int64_t n, int s, const void *B, void *C);

/* ---- blocked dense multiplication (Theorem 2, Section 4.1) ----
 *
 * C (N x N) = A (N x N) * B (N x N), composed of the (N/s)^2 unit calls
 * C_{i,j} = A_i * B_{i,j} (A_i: the i-th N x s vertical strip of A; B_{i,j}:
 * the s x s block in block row i, block column j of B) and the summation
 * of output strip j over i.  The calls are fused into one launch: every
 * output tile receives the contributions of all N/s calls in registers, and
 * no partial product C_{i,j} is written to memory.
 *   A, B: device pointers, N*N input elements each, row-major.
 *   C: device pointer, N*N output elements, row-major, overwritten.
 *   N: order; s <= N <= TCU_MAX_ORDER and N % s == 0, s = tcu_get_unit().
 * Errors: as tcu_mm_tall, with TCU_ERR_SHAPE for N < s or N % s != 0.
 * On success the logical call counter advances by (N/s)^2 = n/m, the number
 * of calls of Theorem 2 (and its lower bound on right-matrix loads). */
int tcu_gemm(const void *A, const void *B, void *C, int64_t N);

/* Stateless forms of the two calls: unit size, dtype and stream are
 * arguments instead of per-thread configuration.  Same contracts, except
 * that s only has to be a supported unit size (16 or 32). */
int tcu_mm_tall_ex(const void *A, int64_t n, int s, const void *B, void *C,
                   int dtype, void *hip_stream);
int tcu_gemm_ex(const void *A, const void *B, void *C, int64_t N, int s,
                int dtype, void *hip_stream);

/* ---- cost accounting (Theorem 2 proof; Section 5 weak model) ----
 * tcu_calls:        logical tensor-unit calls issued (1 per tall call,
 *                   (N/s)^2 per tcu_gemm).
 * tcu_square_calls: the same work counted as s x s calls of the weak model
 *                   (Section 5: a tall call is ceil(n/s) square calls).
 * tcu_work:         sum over calls of n*s, the O(n sqrt(m)) term of each
 *                   call's model time (latency l excluded).
 * tcu_reset_calls:  zero all three. */
int64_t tcu_calls(void);
int64_t tcu_square_calls(void);
int64_t tcu_work(void);
void tcu_reset_calls(void);

/* Static, human-readable text for a status code. */
const char *tcu_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* TCU_H */
