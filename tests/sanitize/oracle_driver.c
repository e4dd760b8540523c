/*
 * Driver for the sanitizer build of the CPU oracle (tests/test_sanitizers.py
 * builds tcu_oracle.c with AddressSanitizer and UndefinedBehaviorSanitizer
 * and links it here).  Calls every exported routine on small inputs,
 * including empty ones, selected rows and rejected arguments, and checks a
 * few exactly known results.  Exit status 0 when all of them hold.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double oracle_f16_to_f64(uint16_t h);
double oracle_bf16_to_f64(uint16_t b);
uint16_t oracle_f64_to_bf16_rne(double x);
void oracle_f64_to_bf16_array(const double *x, uint16_t *out, int64_t count);
void oracle_decode_array(int dtype, const void *in, double *out, int64_t count);
int oracle_mm_f64(int dtype, const void *A, const void *B, int64_t rows, int64_t K, int64_t cols,
                  const int64_t *row_ids, int64_t n_ids, double *C);
int oracle_mm_i64(const int8_t *A, const int8_t *B, int64_t rows, int64_t K, int64_t cols,
                  const int64_t *row_ids, int64_t n_ids, int64_t *C);
int oracle_poly_eval(int dtype, const void *coef, int64_t n, const void *pts, int64_t p,
                     double *value, double *magnitude);
int oracle_transitive_closure(const uint8_t *d, int64_t n, uint8_t *out);
int oracle_dft_direct(const double *x, int64_t n, int64_t batch, double *y);
int oracle_dft_direct_at(const double *x, int64_t n, int64_t batch, const int64_t *ks,
                         int64_t nk, double *y);
int oracle_threads(void);

static int failures = 0;
#define CHECK(c)                                              \
    do {                                                      \
        if (!(c)) {                                           \
            fprintf(stderr, "line %d: %s\n", __LINE__, #c); \
            ++failures;                                       \
        }                                                     \
    } while (0)

int main(void)
{
    /* decoders and the encoder on every pattern and on special values */
    for (uint32_t h = 0; h < 65536; ++h) {
        const double f = oracle_f16_to_f64((uint16_t)h), b = oracle_bf16_to_f64((uint16_t)h);
        if (!isnan(b)) CHECK(oracle_f64_to_bf16_rne(b) == (uint16_t)h);
        (void)f;
    }
    CHECK(oracle_f64_to_bf16_rne(INFINITY) == 0x7f80);
    CHECK(oracle_f64_to_bf16_rne(1e300) == 0x7f80);
    CHECK(oracle_f64_to_bf16_rne(1e-300) == 0);
    CHECK(oracle_f64_to_bf16_rne(NAN) == 0x7fc0);
    double xs[3] = {1.0, -2.0, 0.0};
    uint16_t enc[3];
    oracle_f64_to_bf16_array(xs, enc, 3);
    CHECK(enc[0] == 0x3f80 && enc[1] == 0xc000 && enc[2] == 0);
    double dec[4];
    const int8_t i8[4] = {-128, -1, 0, 127};
    oracle_decode_array(2, i8, dec, 4);
    CHECK(dec[0] == -128.0 && dec[3] == 127.0);

    /* products: 3 x 5 times 5 x 2, all rows and selected rows; empty K */
    uint16_t A[15], B[10];
    int8_t Ai[15], Bi[10];
    for (int i = 0; i < 15; ++i) { A[i] = oracle_f64_to_bf16_rne(i - 7); Ai[i] = (int8_t)(i - 7); }
    for (int i = 0; i < 10; ++i) { B[i] = oracle_f64_to_bf16_rne(3 - i); Bi[i] = (int8_t)(3 - i); }
    double C[6];
    int64_t Ci[6];
    CHECK(oracle_mm_f64(1, A, B, 3, 5, 2, NULL, 3, C) == 0);
    CHECK(oracle_mm_i64(Ai, Bi, 3, 5, 2, NULL, 3, Ci) == 0);
    for (int i = 0; i < 6; ++i) CHECK(C[i] == (double)Ci[i]);
    const int64_t rows[2] = {2, 0};
    double Cs[4];
    CHECK(oracle_mm_f64(1, A, B, 3, 5, 2, rows, 2, Cs) == 0);
    CHECK(Cs[0] == C[4] && Cs[1] == C[5] && Cs[2] == C[0]);
    const int64_t bad_rows[1] = {3};
    CHECK(oracle_mm_f64(1, A, B, 3, 5, 2, bad_rows, 1, Cs) == -1);
    CHECK(oracle_mm_i64(Ai, Bi, 3, 5, 2, bad_rows, 1, Ci) == -1);
    CHECK(oracle_mm_f64(1, A, B, 3, 0, 2, NULL, 3, C) == 0 && C[5] == 0.0);
    CHECK(oracle_mm_f64(7, A, B, 3, 5, 2, NULL, 3, C) == -1);

    /* polynomial: (1 + x)^2 at x = 3 is 16; empty polynomial is 0 */
    const uint16_t coef[3] = {0x3f80, 0x4000, 0x3f80}, pt[2] = {0x4040, 0};
    double val[2], mag[2];
    CHECK(oracle_poly_eval(1, coef, 3, pt, 2, val, mag) == 0);
    CHECK(val[0] == 16.0 && mag[0] == 16.0 && val[1] == 1.0);
    CHECK(oracle_poly_eval(1, coef, 0, pt, 2, val, mag) == 0 && val[0] == 0.0);
    CHECK(oracle_poly_eval(2, coef, 3, pt, 2, val, mag) == -1);

    /* closure: path 0 -> 1 -> 2 on 70 vertices (rows span two words) */
    enum { NV = 70 };
    uint8_t *d = calloc(NV * NV, 1), *out = calloc(NV * NV, 1);
    d[0 * NV + 1] = 1;
    d[1 * NV + 2] = 5;
    d[69 * NV + 69] = 1;
    CHECK(oracle_transitive_closure(d, NV, out) == 0);
    CHECK(out[0 * NV + 2] == 1 && out[2 * NV + 0] == 0 && out[69 * NV + 69] == 1 &&
          out[0 * NV + 0] == 0);
    CHECK(oracle_transitive_closure(d, 0, out) == 0);
    free(d);
    free(out);

    /* DFT: impulse -> all ones; sampled outputs equal the full transform */
    enum { ND = 16 };
    double x[2 * ND * 2], y[2 * ND * 2], ys[2 * 2 * 3];
    memset(x, 0, sizeof(x));
    x[0] = 1.0;
    for (int j = 0; j < ND; ++j) x[2 * ND + 2 * j] = (double)j;
    CHECK(oracle_dft_direct(x, ND, 2, y) == 0);
    for (int k = 0; k < ND; ++k) CHECK(y[2 * k] == 1.0 && y[2 * k + 1] == 0.0);
    const int64_t ks[3] = {0, 8, 15};
    CHECK(oracle_dft_direct_at(x, ND, 2, ks, 3, ys) == 0);
    for (int b = 0; b < 2; ++b)
        for (int t = 0; t < 3; ++t) {
            CHECK(ys[2 * (b * 3 + t)] == y[2 * (b * ND + ks[t])]);
            CHECK(ys[2 * (b * 3 + t) + 1] == y[2 * (b * ND + ks[t]) + 1]);
        }
    const int64_t bad_k[1] = {16};
    CHECK(oracle_dft_direct_at(x, ND, 2, bad_k, 1, ys) == -1);
    CHECK(oracle_dft_direct(x, 0, 1, y) == -1);
    CHECK(oracle_threads() >= 1);

    printf("oracle driver: %d failures\n", failures);
    return failures ? 1 : 0;
}
