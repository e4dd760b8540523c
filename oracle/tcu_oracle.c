/*
 * CPU oracle for the (m,l)-TCU hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  The GPU library never links, calls or includes it,
 * and this file includes nothing from the GPU library.
 *
 * What it computes.  Both calls of the hot path produce the classical matrix
 * product  C[r][j] = sum_k A[r][k] * B[k][j]:
 *   - the native tensor-unit call multiplies an n x sqrt(m) matrix by a
 *     sqrt(m) x sqrt(m) matrix (Section 3, the (m,l)-TCU model definition;
 *     entry notation a_{i,j} from Section 2.2);
 *   - the blocked dense multiplication of Theorem 2 (Section 4.1) splits A
 *     into vertical strips and B into square blocks, but only reorders
 *     semiring operations, so its result is again exactly A*B.
 * The oracle is therefore that plain definition, evaluated in the natural
 * order k = 0, 1, ..., K-1 for every output entry:
 *   - 16-bit floating-point inputs are decoded to binary64 by decoders
 *     written here from the IEEE 754 binary16 and bfloat16 format
 *     definitions; a product of two such values is exact in binary64 and
 *     the running sum is kept in binary64;
 *   - int8 inputs are widened to int64 and summed exactly.
 * A bfloat16 output is produced by one round-to-nearest-even step applied
 * directly to the binary64 sum (no intermediate binary32 rounding).
 *
 * Precision is not fixed by the paper (Section 3.1 leaves limited precision
 * out of the model), so binary64 / int64 is the oracle's arithmetic.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F16 = 0, ORC_BF16 = 1, ORC_I8 = 2 };

/* ---------------------------------------------------------------- decoders */

/* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction
 * bits.  Exponent field 0 encodes zero/subnormals (value frac * 2^-24),
 * field 31 encodes infinities (frac == 0) and NaNs. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expf = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expf == 0)
        v = ldexp((double)frac, -24);
    else if (expf == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + frac), expf - 25);
    return sign ? -v : v;
}

/* bfloat16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits.
 * Exponent field 0 encodes zero/subnormals (value frac * 2^-133),
 * field 255 encodes infinities (frac == 0) and NaNs. */
double oracle_bf16_to_f64(uint16_t b)
{
    int sign = (b >> 15) & 1;
    int expf = (b >> 7) & 0xff;
    int frac = b & 0x7f;
    double v;
    if (expf == 0)
        v = ldexp((double)frac, -133);
    else if (expf == 255)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(128 + frac), expf - 134);
    return sign ? -v : v;
}

/* ----------------------------------------------------------------- encoder */

/* Round a binary64 value to the nearest bfloat16, ties to the value whose
 * last fraction bit is 0, in one step.  Values whose magnitude rounds to
 * 2^128 or beyond become infinity; NaN becomes the quiet NaN 0x7fc0 with
 * the input's sign. */
uint16_t oracle_f64_to_bf16_rne(double x)
{
    uint16_t sign = signbit(x) ? 0x8000 : 0;
    if (isnan(x))
        return sign | 0x7fc0;
    double ax = fabs(x);
    if (isinf(ax))
        return sign | 0x7f80;
    if (ax == 0.0)
        return sign;

    /* ax = f * 2^e with f in [0.5, 1), so ax lies in [2^(e-1), 2^e). */
    int e;
    (void)frexp(ax, &e);
    int binade = e - 1;           /* ax in [2^binade, 2^(binade+1)) */
    if (binade < -126)
        binade = -126;            /* subnormal range shares the 2^-133 spacing */
    int ulp_exp = binade - 7;     /* spacing of bfloat16 values there */

    double q = ldexp(ax, -ulp_exp);   /* exact: scaling by a power of two */
    double fl = floor(q);
    double rem = q - fl;              /* exact */
    double k;
    if (rem > 0.5)
        k = fl + 1.0;
    else if (rem < 0.5)
        k = fl;
    else
        k = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;

    double r = ldexp(k, ulp_exp);
    if (r >= ldexp(1.0, 128))
        return sign | 0x7f80;
    if (r < ldexp(1.0, -126)) {
        /* subnormal (or the smallest normal when k reached 128) */
        uint16_t frac = (uint16_t)ldexp(r, 133);
        return sign | frac;
    }
    int er;
    double fr = frexp(r, &er);        /* r = fr * 2^er, fr in [0.5, 1) */
    uint16_t expf = (uint16_t)(er - 1 + 127);
    uint16_t frac = (uint16_t)(ldexp(fr, 8) - 128.0);
    return sign | (uint16_t)(expf << 7) | frac;
}

void oracle_f64_to_bf16_array(const double *x, uint16_t *out, int64_t count)
{
    for (int64_t i = 0; i < count; ++i)
        out[i] = oracle_f64_to_bf16_rne(x[i]);
}

void oracle_decode_array(int dtype, const void *in, double *out, int64_t count)
{
    for (int64_t i = 0; i < count; ++i) {
        if (dtype == ORC_F16)
            out[i] = oracle_f16_to_f64(((const uint16_t *)in)[i]);
        else if (dtype == ORC_BF16)
            out[i] = oracle_bf16_to_f64(((const uint16_t *)in)[i]);
        else
            out[i] = (double)((const int8_t *)in)[i];
    }
}

/* ------------------------------------------------------------------ product */

static double decode_one(int dtype, const void *p, int64_t idx)
{
    if (dtype == ORC_F16)
        return oracle_f16_to_f64(((const uint16_t *)p)[idx]);
    return oracle_bf16_to_f64(((const uint16_t *)p)[idx]);
}

/* C[t][j] = sum_{k<K} A[r_t][k] * B[k][j] in binary64, for floating-point
 * inputs (dtype ORC_F16 or ORC_BF16).
 *   A: rows x K, row-major; B: K x cols, row-major.
 *   row_ids: the rows r_t of A whose products are wanted (n_ids of them),
 *            or NULL for all rows (then n_ids must equal rows).
 *   C: n_ids x cols, row-major binary64, written.
 * Returns 0, or -1 for a bad argument. */
int oracle_mm_f64(int dtype, const void *A, const void *B,
                  int64_t rows, int64_t K, int64_t cols,
                  const int64_t *row_ids, int64_t n_ids, double *C)
{
    if ((dtype != ORC_F16 && dtype != ORC_BF16) || !A || !B || !C ||
        rows < 0 || K < 0 || cols < 0 || n_ids < 0)
        return -1;
    if (!row_ids && n_ids != rows)
        return -1;
    if (row_ids)
        for (int64_t t = 0; t < n_ids; ++t)
            if (row_ids[t] < 0 || row_ids[t] >= rows)
                return -1;

    double *Bd = (double *)malloc(sizeof(double) * (size_t)(K * cols > 0 ? K * cols : 1));
    if (!Bd)
        return -1;
    for (int64_t i = 0; i < K * cols; ++i)
        Bd[i] = decode_one(dtype, B, i);

#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < n_ids; ++t) {
        int64_t r = row_ids ? row_ids[t] : t;
        double *c = C + t * cols;
        for (int64_t j = 0; j < cols; ++j)
            c[j] = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double a = decode_one(dtype, A, r * K + k);
            const double *b = Bd + k * cols;
            for (int64_t j = 0; j < cols; ++j)
                c[j] += a * b[j];
        }
    }
    free(Bd);
    return 0;
}

/* Same contract for int8 inputs, summed exactly in int64. */
int oracle_mm_i64(const int8_t *A, const int8_t *B,
                  int64_t rows, int64_t K, int64_t cols,
                  const int64_t *row_ids, int64_t n_ids, int64_t *C)
{
    if (!A || !B || !C || rows < 0 || K < 0 || cols < 0 || n_ids < 0)
        return -1;
    if (!row_ids && n_ids != rows)
        return -1;
    if (row_ids)
        for (int64_t t = 0; t < n_ids; ++t)
            if (row_ids[t] < 0 || row_ids[t] >= rows)
                return -1;

#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < n_ids; ++t) {
        int64_t r = row_ids ? row_ids[t] : t;
        int64_t *c = C + t * cols;
        for (int64_t j = 0; j < cols; ++j)
            c[j] = 0;
        for (int64_t k = 0; k < K; ++k) {
            int64_t a = A[r * K + k];
            const int8_t *b = B + k * cols;
            for (int64_t j = 0; j < cols; ++j)
                c[j] += a * (int64_t)b[j];
        }
    }
    return 0;
}

/* Threads an OpenMP region of this library runs with. */
int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------ batch polynomial evaluation */
/*
 * Theorem 11 (Section 4.8) evaluates A(x) = sum_{h<n} a_h x^h at p points.
 * Its method (power matrix X times the coefficient matrix in unit-sized
 * blocks, then a combine over the blocks' columns) only regroups that sum,
 * so the oracle is the definition itself: for every point, the terms
 * a_h * x^h for h = 0, 1, ..., n-1 in that order, the power kept by the
 * recurrence x^0 = 1, x^(h+1) = x^h * x, everything in binary64 on the
 * decoded 16-bit inputs.  It also returns the magnitude sum
 * sum_h |a_h| |x|^h that bounds the rounding error of any evaluation.
 */
int oracle_poly_eval(int dtype, const void *coef, int64_t n, const void *pts, int64_t p,
                     double *value, double *magnitude)
{
    if (dtype != ORC_F16 && dtype != ORC_BF16) return -1;
    if (n < 0 || p < 0) return -1;
    double *a = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    if (!a) return -2;
    for (int64_t h = 0; h < n; ++h) a[h] = decode_one(dtype, coef, h);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < p; ++i) {
        const double x = decode_one(dtype, pts, i);
        double power = 1.0, sum = 0.0, mag = 0.0;
        for (int64_t h = 0; h < n; ++h) {
            sum += a[h] * power;
            mag += fabs(a[h]) * fabs(power);
            power *= x;
        }
        value[i] = sum;
        magnitude[i] = mag;
    }
    free(a);
    return 0;
}

/* ---------------------------------------------------- transitive closure */
/*
 * Transitive closure of a directed graph (Section 4.3): from the n x n 0/1
 * adjacency matrix d, c[i][j] = 1 iff j is reachable from i by a path of one
 * or more edges.  The oracle is the iterative algorithm the section starts
 * from, d[i][j] <- d[i][j] OR (d[i][k] AND d[k][j]) for k, then i, then j,
 * updating d in place.  Rows are held as bit sets (bit j of row i), so the
 * innermost j loop ORs row k into row i one 64-bit word at a time whenever
 * d[i][k] = 1 -- the same loop order and the same updates.
 *   d: n*n bytes, row-major, 0 = no edge, anything else = edge (read);
 *   out: n*n bytes, the closure as 0/1 (written).
 */
int oracle_transitive_closure(const uint8_t *d, int64_t n, uint8_t *out)
{
    if (n < 0) return -1;
    const int64_t words = (n + 63) / 64;
    uint64_t *bits = (uint64_t *)calloc((size_t)(n > 0 ? n * words : 1), sizeof(uint64_t));
    if (!bits) return -2;
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j)
            if (d[i * n + j]) bits[i * words + j / 64] |= (uint64_t)1 << (j % 64);
    for (int64_t k = 0; k < n; ++k) {
        const uint64_t *rk = bits + k * words;
        const uint64_t kbit = (uint64_t)1 << (k % 64);
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            uint64_t *ri = bits + i * words;
            if (ri[k / 64] & kbit)
                for (int64_t w = 0; w < words; ++w) ri[w] |= rk[w];
        }
    }
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j)
            out[i * n + j] = (uint8_t)((bits[i * words + j / 64] >> (j % 64)) & 1u);
    free(bits);
    return 0;
}

/* ----------------------------------------------- discrete Fourier transform */
/*
 * Section 4.5 defines the DFT of an n-vector x as y = x^T W with the Fourier
 * matrix W[r][c] = exp(-2 pi i r c / n).  This is that definition, one
 * output at a time: y[k] = sum_j x[j] (cos t - i sin t), t = 2 pi (j k mod n)
 * / n, in binary64 (the product j k is reduced mod n exactly in integers
 * first).  x, y: batch * n complex values as interleaved (re, im) doubles.
 * O(n^2) per vector: for checking small sizes and for pinning.
 */
int oracle_dft_direct(const double *x, int64_t n, int64_t batch, double *y)
{
    if (n < 1 || batch < 0) return -1;
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t k = 0; k < n; ++k) {
            const double *xb = x + 2 * b * n;
            double re = 0.0, im = 0.0;
            for (int64_t j = 0; j < n; ++j) {
                const int64_t e = (int64_t)(((unsigned __int128)j * (unsigned __int128)k) % (unsigned __int128)n);
                const double t = two_pi * (double)e / (double)n;
                const double c = cos(t), s = sin(t);
                /* (xr + i xi)(c - i s) */
                re += xb[2 * j] * c + xb[2 * j + 1] * s;
                im += xb[2 * j + 1] * c - xb[2 * j] * s;
            }
            y[2 * (b * n + k)] = re;
            y[2 * (b * n + k) + 1] = im;
        }
    return 0;
}

/*
 * The same definition of Section 4.5 at chosen output frequencies only:
 * y[b][t] = sum_j x_b[j] exp(-2 pi i j k_t / n) for the nk frequencies
 * k_t in ks (each 0 <= k_t < n), in binary64, the exponent j k_t reduced
 * mod n exactly in integers as above.  O(n) per frequency, so vectors of
 * any length can be checked on a sample of their outputs.
 *   x: batch * n complex values (interleaved re, im doubles);
 *   y: batch * nk complex values, row b holding the nk sampled outputs.
 */
int oracle_dft_direct_at(const double *x, int64_t n, int64_t batch, const int64_t *ks,
                         int64_t nk, double *y)
{
    if (n < 1 || batch < 0 || nk < 0 || (nk > 0 && !ks)) return -1;
    for (int64_t t = 0; t < nk; ++t)
        if (ks[t] < 0 || ks[t] >= n) return -1;
    const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t b = 0; b < batch; ++b)
        for (int64_t t = 0; t < nk; ++t) {
            const double *xb = x + 2 * b * n;
            const int64_t k = ks[t];
            double re = 0.0, im = 0.0;
            for (int64_t j = 0; j < n; ++j) {
                const int64_t e = (int64_t)(((unsigned __int128)j * (unsigned __int128)k) % (unsigned __int128)n);
                const double th = two_pi * (double)e / (double)n;
                const double c = cos(th), s = sin(th);
                re += xb[2 * j] * c + xb[2 * j + 1] * s;
                im += xb[2 * j + 1] * c - xb[2 * j] * s;
            }
            y[2 * (b * nk + t)] = re;
            y[2 * (b * nk + t) + 1] = im;
        }
    return 0;
}
