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
 *   - tcu_gemm_rect: the same decomposition for rectangular, strided and
 *     accumulating products (Corollary 1; the D functions' update).
 *   - tcu_transitive_closure: the blocked transitive closure (Theorem 5).
 *   - tcu_dft: the discrete Fourier transform by Cooley-Tukey (Theorem 7).
 *   - tcu_poly_eval: batch polynomial evaluation (Theorem 11).
 *
 * Throughout, s = sqrt(m) is the unit size (a machine parameter of the
 * model), n is the row count of a tall call and N the order of the square
 * product.
 *
 * Conventions shared by every entry point:
 *   - All matrix pointers are DEVICE pointers (memory of the current HIP
 *     device).  Matrices are row-major; element (r, c) of an R x C matrix
 *     is at index r*ld + c, with ld = C (contiguous) except where an entry
 *     point takes an explicit row pitch ld (tcu_gemm_rect).
 *   - The caller allocates and frees A, B and C.  The library never
 *     allocates, frees or retains them, and keeps no pointer across calls.
 *   - C is overwritten with the product (the unit stores its result), except
 *     in the accumulating form of tcu_gemm_rect.
 *   - Calls are asynchronous on the stream in effect; the caller synchronises.
 *   - Every call returns a tcu_status: 0 on success, a negative code on
 *     failure.  Argument checks (null, shape, unit size, dtype, alignment,
 *     overlap) all run before any HIP call, so a rejected call touches no
 *     device state.  A rejected call leaves C unmodified and does not count
 *     as a tensor-unit call.
 *   - The library cannot tell a device pointer from a host or stale one by
 *     its value: a kernel given such a pointer faults the GPU.  With pointer
 *     checks on (TCU_KNOB_CHECK_POINTERS, or the environment variable
 *     TCU_DEBUG set to a nonzero integer when the library is loaded), every
 *     entry point first asks the HIP runtime whether each operand's whole
 *     extent lies inside one device allocation of the current device, and
 *     returns TCU_ERR_POINTER, before any launch, if not.  The check costs a
 *     few runtime queries per call and is off by default.
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
    TCU_ERR_NO_DEVICE = -7,   /* no HIP device is visible */
    TCU_ERR_POINTER = -8,     /* pointer checks on: an operand is not inside one device
                                 allocation of the current device (tcu_check_device_range) */
    TCU_ERR_SCRATCH = -9      /* the problem needs more than the fixed scratch of an
                                 allocation-free entry point (tcu_dft_noalloc) */
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
 * of calls of Theorem 2 (and its lower bound on right-matrix loads).
 * Reproducibility: int32 and bfloat16 results are the same on every call.
 * A binary32 result is too, unless the product splits the contracted index
 * across workgroups -- which it does when the 256 x 256 output tiles are
 * fewer than the device's compute units, or when they do not fill a whole
 * number of rounds of the persistent grid (the tiles of the last round are
 * then split) -- because the partial sums are then added into C with atomic
 * additions in no fixed order: the low bits of such a binary32 result may
 * differ from call to call (each result is within the stated summation
 * bound; the order-8192 products are not split). */
int tcu_gemm(const void *A, const void *B, void *C, int64_t N);

/* Stateless forms of the two calls: unit size, dtype and stream are
 * arguments instead of per-thread configuration.  Same contracts, except
 * that s only has to be a supported unit size (16 or 32). */
int tcu_mm_tall_ex(const void *A, int64_t n, int s, const void *B, void *C,
                   int dtype, void *hip_stream);
int tcu_gemm_ex(const void *A, const void *B, void *C, int64_t N, int s,
                int dtype, void *hip_stream);

/* ---- rectangular, strided and accumulating product ----
 *
 * C (M x N) = A (M x K) * B (K x N)                      (flags = 0)
 * C (M x N) = C + A (M x K) * B (K x N)                  (flags = TCU_ACCUMULATE)
 *
 * Corollary 1 (Section 4.1) multiplies a sqrt(n) x r matrix by an
 * r x sqrt(n) one by cutting it into unit-sized pieces and applying
 * Theorem 2.  This entry point does exactly that for any M, K, N: A is cut
 * into M x s vertical strips A_i (i < ceil(K/s)), B into s x s blocks
 * B_{i,j} (j < ceil(N/s)), and output strip j is sum_i A_i * B_{i,j}, so
 * it issues ceil(K/s) * ceil(N/s) tall calls with n = M rows (the bound
 * r*sqrt(n)/m of Corollary 1 when M = N = sqrt(n), K = r).  Dimensions
 * that are not multiples of s are zero-padded: the missing rows and columns
 * of the last strip and blocks are taken as zeros, which leaves the
 * product unchanged; nothing outside the M x N output is written.
 * The accumulating form is the update X <- X + Y * Z that the D functions
 * of the Gaussian-elimination and transitive-closure algorithms
 * (Sections 4.2 and 4.3) ask of the unit.
 *
 *   A: M x K input elements, row r at A + r*lda elements (lda >= K).
 *   B: K x N input elements, row k at B + k*ldb elements (ldb >= N).
 *   C: M x N output elements, row r at C + r*ldc elements (ldc >= N); read
 *      too when accumulating.  The three matrices may be views into larger
 *      row-major arrays.
 *   M, K, N: 0 <= M, K, N <= TCU_MAX_RECT_DIM.  M = 0 or N = 0 is a no-op;
 *      K = 0 writes zeros (flags = 0) or leaves C unchanged (accumulate).
 *   flags: 0 or TCU_ACCUMULATE.
 * A, B or C may be NULL when that matrix has no elements (M*K, K*N or M*N
 * is 0); otherwise NULL is TCU_ERR_NULL.
 * Arithmetic: the sum over K is formed in binary32 (int32 for int8
 * inputs); when accumulating, the stored C value is added to it in the
 * same type and the result is stored once (rounded to nearest even for a
 * bfloat16 output).  For int8 inputs K < 2^17 is required, so A*B is exact
 * in int32; the accumulated C + A*B wraps modulo 2^32 if it leaves the
 * int32 range.  As for tcu_gemm, a binary32 result whose contracted index
 * is split across workgroups (few output tiles with a long K, or the tiles
 * of a partial last round) is summed in no fixed order, so its low bits may
 * differ from call to call; int32 and bfloat16 results are reproducible.
 * Layout rules: base pointers 16-byte aligned; every element each operand
 * addresses must lie below 2^40 bytes from its base.  Row pitches need no
 * alignment, but pitches whose byte size is a multiple of 16 (lda, ldb, ldc
 * multiples of 8 for 16-bit, of 16 for int8, of 4 for 32-bit elements) take
 * the vector-load kernels; others use element-wise loads.  C must not share
 * an element with A or B: views of one array with the same byte pitch are
 * checked element-exactly, other cases by address range.
 * Errors: TCU_ERR_NULL, TCU_ERR_SHAPE (a dimension out of range, int8 with
 * K >= 2^17, a pitch below its row length, an extent of 2^40 bytes or more),
 * TCU_ERR_UNSUPPORTED (unit size, dtype or flags), TCU_ERR_ALIGN,
 * TCU_ERR_OVERLAP, TCU_ERR_NO_DEVICE, TCU_ERR_HIP.
 * Cost accounting: ceil(K/s)*ceil(N/s) calls, each of ceil(M/s) square
 * calls and ceil(M/s)*s*s work (0 of each if M, K or N is 0). */
#define TCU_ACCUMULATE 1
#define TCU_MAX_RECT_DIM ((int64_t)1 << 30)
int tcu_gemm_rect(const void *A, int64_t lda, const void *B, int64_t ldb, void *C, int64_t ldc,
                  int64_t M, int64_t K, int64_t N, int flags);
int tcu_gemm_rect_ex(const void *A, int64_t lda, const void *B, int64_t ldb, void *C,
                     int64_t ldc, int64_t M, int64_t K, int64_t N, int flags, int s, int dtype,
                     void *hip_stream);

/* ---- batch polynomial evaluation (Theorem 11, Section 4.8) ----
 *
 * out[i] = A(points[i]) = sum_{h<n} coef[h] * points[i]^h, for 0 <= i < p.
 *
 * Theorem 11's method: the p x s matrix X of the powers x_i^0 .. x_i^(s-1),
 * times the s x (n/s) matrix whose column j holds a_(js) .. a_(js+s-1)
 * (the coefficients read column-major), cut into s x s blocks -- ceil(n/m)
 * tall calls of p rows -- followed by A(x_i) = sum_j C[i][j] x_i^(js).
 * The powers are formed in binary32 and handed to the unit as the sum of
 * two bfloat16 words (X = X_hi + X_lo, about 2^-17 relative accuracy), so
 * every call is issued twice; binary16 coefficients are split exactly into
 * two bfloat16 words each (c = c_hi + c_lo), so with binary16 inputs every
 * call is issued four times -- bfloat16 has binary32's exponent range, so
 * small powers x^k do not underflow as binary16 words would.  The combine
 * runs in binary32 and C is never stored.  n and p need not be multiples of
 * s (zero padding; the theorem assumes them).
 *   coef: n input elements (binary16 or bfloat16, the unit's input type).
 *   n: number of coefficients (degree n-1); 0 <= n <= TCU_MAX_ROWS; n = 0
 *      gives zeros.
 *   points: p input elements (same type); 0 <= p <= TCU_MAX_ROWS; p = 0 is
 *      a no-op.
 *   out: p output elements: binary32 (TCU_F16_F32, TCU_BF16_F32) or
 *      bfloat16 rounded once to nearest even (TCU_BF16_BF16).
 * The unit size and dtype come from tcu_get_unit() / tcu_get_dtype()
 * (TCU_I8_I32 is TCU_ERR_UNSUPPORTED).  Results are meaningful while
 * |x|^(n-1) and the partial sums stay in binary32's normal range (the
 * theorem assumes evaluation without overflow; a term a_h x^h whose powers
 * fall below about 2^-118 loses relative accuracy to binary32 and bfloat16
 * underflow).
 * A pointer may be NULL only if its array is empty.  Errors: TCU_ERR_NULL,
 * TCU_ERR_SHAPE, TCU_ERR_UNSUPPORTED, TCU_ERR_ALIGN (16-byte base
 * alignment), TCU_ERR_OVERLAP (out overlapping coef or points),
 * TCU_ERR_NO_DEVICE, TCU_ERR_HIP.
 * Cost accounting: 2*ceil(n/m) calls (4*ceil(n/m) for binary16 inputs)
 * of ceil(p/s) square calls each. */
int tcu_poly_eval(const void *coef, int64_t n, const void *points, int64_t p, void *out);
int tcu_poly_eval_ex(const void *coef, int64_t n, const void *points, int64_t p, void *out, int s,
                     int dtype, void *hip_stream);

/* ---- transitive closure (Theorem 5, Section 4.3) ----
 *
 * X <- the transitive closure of the directed graph whose n x n adjacency
 * matrix X holds: afterwards X[i][j] = 1 iff vertex j is reachable from
 * vertex i by a path of one or more edges, else 0.  In place.
 *   X: n x n int8 entries, row i at X + i*ld bytes (ld >= n); on input any
 *      nonzero byte is an edge (self loops allowed); on output 0 or 1.
 *   n: number of vertices, 0 <= n <= TCU_MAX_RECT_DIM (n = 0 is a no-op);
 *      need not be a multiple of s.
 * The section's blocked algorithm: per pivot block, close the diagonal
 * block (A), update the pivot block row and column through it (B, C), then
 * every other block by the D function X_ij <- min(X_ij + X_ik X_kj, 1) on the
 * int8 matrix cores.  Pivot blocks here are 256 vertices wide.
 * The unit size comes from tcu_get_unit() (it sets the cost accounting);
 * the stream from tcu_get_stream().  Errors: TCU_ERR_NULL, TCU_ERR_SHAPE
 * (n out of range, ld < n, extent of 2^40 bytes or more),
 * TCU_ERR_UNSUPPORTED, TCU_ERR_ALIGN (X not 16-byte aligned),
 * TCU_ERR_NO_DEVICE, TCU_ERR_HIP.
 * Cost accounting (the s-blocked algorithm): q(q-1) calls of the D function
 * with q = ceil(n/s), each of (q-1) square calls. */
int tcu_transitive_closure(void *X, int64_t n, int64_t ld);
int tcu_transitive_closure_ex(void *X, int64_t n, int64_t ld, int s, void *hip_stream);

/* ---- discrete Fourier transform (Theorem 7, Section 4.5) ----
 *
 * y_b[k] = sum_{j<n} x_b[j] exp(-2 pi i j k / n), for b < batch: the DFT
 * y = x^T W of each vector, W[r][c] = exp(-2 pi i r c / n).
 * The section's Cooley-Tukey recursion with radix s = sqrt(m): per level,
 * the DFTs of length s of n/s interleaved subsequences as the tall product
 * X^T W_s (n/s rows through the unit), the twiddles w^(r c) and the
 * transpose, for ceil(log_s n) levels (the last of radix n/s^(L-1) <= s).
 * Complex products are real products on the unit; data and W enter as
 * hi + lo bfloat16 words (about 2^-16 relative accuracy per level).
 *   x: batch * n complex values, each two binary32 (re, im), vector b at
 *      x + 2 b n floats; read only.
 *   y: batch * n complex values, written; must not overlap x or work.
 *   work: batch * n complex values of scratch the levels alternate through
 *      (its contents are overwritten); must not overlap x or y; may be NULL
 *      when n <= s (one level).
 *   n: a power of two, 1 <= n <= TCU_MAX_DFT_N; batch >= 0 (0: no-op).
 * The unit size and stream come from tcu_get_unit() / tcu_get_stream().
 * Errors: TCU_ERR_NULL, TCU_ERR_SHAPE (n not a power of two or out of range,
 * batch < 0, extent of 2^40 bytes or more), TCU_ERR_UNSUPPORTED,
 * TCU_ERR_ALIGN (16-byte base alignment), TCU_ERR_OVERLAP,
 * TCU_ERR_NO_DEVICE, TCU_ERR_HIP.
 * Cost accounting: per vector and level, 4 calls (the complex product as
 * four real ones) of n/R rows, R the level's radix. */
#define TCU_MAX_DFT_N ((int64_t)1 << 30)
int tcu_dft(const void *x, void *y, void *work, int64_t n, int64_t batch);
int tcu_dft_ex(const void *x, void *y, void *work, int64_t n, int64_t batch, int s,
               void *hip_stream);

/* ---- the DFT without a caller-supplied work buffer ----
 *
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * transform as tcu_dft_ex, with the levels' second buffer taken from a
 * fixed array of TCU_DFT_NOALLOC_MAX_BYTES bytes of device memory that the
 * library holds on each device it runs on, from its first use there until
 * the process ends.  The call itself allocates nothing.
 *   x, y, n, batch, s, hip_stream: as tcu_dft_ex (y must not overlap x).
 *   When the transform has more than one level (n > s), batch * n * 8 bytes
 *   must not exceed TCU_DFT_NOALLOC_MAX_BYTES, else TCU_ERR_SCRATCH and
 *   nothing is launched; one level needs no scratch and has no such limit.
 * Every call on a device shares that device's array and leaves its
 * contents behind (the levels overwrite it before reading it, so nothing is
 * cleared): calls that overlap in time on one device -- on different
 * streams, or from different host threads -- race on it and must be
 * serialized by the caller.
 * Errors: as tcu_dft_ex, plus TCU_ERR_SCRATCH.  Cost accounting: as tcu_dft. */
#define TCU_DFT_NOALLOC_MAX_BYTES ((int64_t)64 << 20)
int tcu_dft_noalloc(const void *x, void *y, int64_t n, int64_t batch, int s, void *hip_stream);

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

/* ---- pointer checks and test overrides ----
 *
 * tcu_check_device_range: TCU_OK if bytes == 0, or if [p, p + bytes) lies
 * inside one device (or managed) allocation of the current HIP device;
 * TCU_ERR_POINTER if p is a host pointer, unknown to the runtime, on
 * another device, or the range runs past its allocation (with torch's
 * caching allocator: past the cached block holding it); TCU_ERR_SHAPE for
 * bytes < 0; TCU_ERR_NO_DEVICE / TCU_ERR_HIP if the runtime cannot answer.
 * A failed query leaves HIP's last-error state as it was before the call.
 * This is the check every entry point applies to each operand while
 * TCU_KNOB_CHECK_POINTERS is 1.
 *
 * tcu_set_knob / tcu_get_knob: process-wide overrides of the library's
 * automatic choices, for tests that must reach every kernel path on small
 * shapes, and the pointer-check switch.  Value 0 restores the automatic
 * choice.  Products never read the environment; only the initial value of
 * TCU_KNOB_CHECK_POINTERS comes from TCU_DEBUG at load time.
 *   TCU_KNOB_GEMM_KERNEL: TCU_PATH_AUTO, TCU_PATH_FULL_TILE (the 256 x 256
 *     persistent kernel wherever its shape conditions hold),
 *     TCU_PATH_GENERAL (the general kernel), TCU_PATH_RING (the small-tile
 *     ring kernel where its shape conditions hold).
 *   TCU_KNOB_PP_GRID: workgroups of the persistent full-tile kernel, in the
 *     products and in the transitive closure's D updates (0: one per compute
 *     unit).
 *   TCU_KNOB_SPLIT_K: forced number of contracted-index ranges of a
 *     full-tile product with binary32/int32 output (0: by size).
 *   TCU_KNOB_TAIL_SPLIT: forced number of ranges of the last round's tiles
 *     (0: by size; 1: none).
 *   TCU_KNOB_CHECK_POINTERS: 1 = check every operand with
 *     tcu_check_device_range before launching, 0 = no checks.
 *   TCU_KNOB_DFT_PAIRS: 1 = every DFT level its own launch; 0 = two
 *     consecutive full-radix levels in one launch where possible (the same
 *     result, bit for bit).
 * Returns TCU_OK, or TCU_ERR_UNSUPPORTED for an unknown knob or a value
 * out of range (the knob is then unchanged); tcu_get_knob returns -1 for an
 * unknown knob.  Changing a knob while another thread issues calls is safe
 * but gives that thread either value. */
enum {
    TCU_KNOB_GEMM_KERNEL = 0,
    TCU_KNOB_PP_GRID = 1,
    TCU_KNOB_SPLIT_K = 2,
    TCU_KNOB_TAIL_SPLIT = 3,
    TCU_KNOB_CHECK_POINTERS = 4,
    TCU_KNOB_DFT_PAIRS = 5
};
enum { TCU_PATH_AUTO = 0, TCU_PATH_FULL_TILE = 1, TCU_PATH_GENERAL = 2, TCU_PATH_RING = 3 };
int tcu_check_device_range(const void *p, int64_t bytes);
int tcu_set_knob(int knob, int value);
int tcu_get_knob(int knob);

#ifdef __cplusplus
}
#endif

#endif /* TCU_H */
