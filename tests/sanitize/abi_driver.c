/*
 * Host-only driver for the sanitizer build of the C ABI's argument
 * validation (tests/test_sanitizers.py builds tcu_abi.cpp with
 * AddressSanitizer and UndefinedBehaviorSanitizer and links it here).
 *
 * Every call uses fake, never-dereferenced device addresses and is built to
 * be rejected by validation, except the calls marked "valid", which reach the
 * device query and must report TCU_ERR_NO_DEVICE: the driver runs only on a
 * machine with no GPU.  Exit status 0 when every status is the expected one.
 */
#include <stdint.h>
#include <stdio.h>

#include "tcu.h"

static int failures = 0;

static void expect(const char *what, int got, int want)
{
    if (got != want) {
        fprintf(stderr, "%s: got %d, want %d\n", what, got, want);
        ++failures;
    }
}

#define PA ((const void *)(uintptr_t)0x10000000u)
#define PB ((const void *)(uintptr_t)0x20000000u)
#define PC ((void *)(uintptr_t)0x30000000u)

int main(void)
{
    const int64_t big = (int64_t)1 << 62;

    /* configuration */
    expect("set_unit 8", tcu_set_unit(8), TCU_ERR_UNSUPPORTED);
    expect("set_unit 32", tcu_set_unit(32), TCU_OK);
    expect("set_dtype 7", tcu_set_dtype(7), TCU_ERR_UNSUPPORTED);
    expect("set_dtype bf16", tcu_set_dtype(TCU_BF16_F32), TCU_OK);
    expect("set_knob bad", tcu_set_knob(9, 1), TCU_ERR_UNSUPPORTED);
    expect("get_knob bad", tcu_get_knob(-3), -1);

    /* native call */
    expect("tall null", tcu_mm_tall_ex(0, 64, 32, PB, PC, 1, 0), TCU_ERR_NULL);
    expect("tall n<s", tcu_mm_tall_ex(PA, 31, 32, PB, PC, 1, 0), TCU_ERR_SHAPE);
    expect("tall n huge", tcu_mm_tall_ex(PA, big, 32, PB, PC, 1, 0), TCU_ERR_SHAPE);
    expect("tall n neg", tcu_mm_tall_ex(PA, -big, 32, PB, PC, 1, 0), TCU_ERR_SHAPE);
    expect("tall align", tcu_mm_tall_ex((const char *)PA + 2, 64, 32, PB, PC, 1, 0),
           TCU_ERR_ALIGN);
    expect("tall overlap", tcu_mm_tall_ex(PA, 64, 32, PB, (void *)PA, 1, 0), TCU_ERR_OVERLAP);
    expect("tall valid", tcu_mm_tall_ex(PA, 64, 32, PB, PC, 1, 0), TCU_ERR_NO_DEVICE);
    expect("tall state s", tcu_mm_tall(PA, 64, 16, PB, PC), TCU_ERR_UNSUPPORTED);

    /* square product */
    expect("gemm N%s", tcu_gemm_ex(PA, PB, PC, 100, 32, 1, 0), TCU_ERR_SHAPE);
    expect("gemm N huge", tcu_gemm_ex(PA, PB, PC, big, 32, 1, 0), TCU_ERR_SHAPE);
    expect("gemm i8 2^17", tcu_gemm_ex(PA, PB, PC, (int64_t)1 << 17, 32, 3, 0), TCU_ERR_SHAPE);
    expect("gemm valid", tcu_gemm_ex(PA, PB, PC, 256, 32, 1, 0), TCU_ERR_NO_DEVICE);

    /* rectangular product: extents near the saturation limits, overlap of
     * views of one array */
    expect("rect pitch < K", tcu_gemm_rect_ex(PA, 10, PB, 64, PC, 64, 64, 64, 64, 0, 32, 1, 0),
           TCU_ERR_SHAPE);
    expect("rect huge pitch",
           tcu_gemm_rect_ex(PA, ((int64_t)1 << 40) - 1, PB, 64, PC, 64, 1 << 30, 64, 64, 0, 32,
                            1, 0),
           TCU_ERR_SHAPE);
    expect("rect dims", tcu_gemm_rect_ex(PA, big, PB, big, PC, big, big, big, big, 0, 32, 1, 0),
           TCU_ERR_SHAPE);
    expect("rect neg", tcu_gemm_rect_ex(PA, 64, PB, 64, PC, 64, -1, 64, 64, 0, 32, 1, 0),
           TCU_ERR_SHAPE);
    expect("rect flags", tcu_gemm_rect_ex(PA, 64, PB, 64, PC, 64, 64, 64, 64, 6, 32, 1, 0),
           TCU_ERR_UNSUPPORTED);
    /* C and A as blocks of one 1024-column bf16 array (pitch 2048 bytes):
     * disjoint blocks pass validation, a shared element is an overlap */
    {
        const char *X = (const char *)PA;
        expect("rect disjoint blocks",
               tcu_gemm_rect_ex(X, 1024, PB, 64, (void *)(X + 256 * 4), 1024, 64, 64, 64, 0, 32,
                                2, 0),
               TCU_ERR_NO_DEVICE);
        expect("rect shared element",
               tcu_gemm_rect_ex(X, 1024, PB, 64, (void *)(X + 63 * 2048 + 96), 1024, 64, 64, 64,
                                0, 32, 2, 0),
               TCU_ERR_OVERLAP);
    }
    expect("rect empty", tcu_gemm_rect_ex(0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 32, 1, 0), TCU_OK);

    /* polynomial evaluation, closure, DFT */
    expect("poly i8", tcu_poly_eval_ex(PA, 10, PB, 10, PC, 32, 3, 0), TCU_ERR_UNSUPPORTED);
    expect("poly neg", tcu_poly_eval_ex(PA, -1, PB, 10, PC, 32, 1, 0), TCU_ERR_SHAPE);
    expect("poly huge", tcu_poly_eval_ex(PA, big, PB, 10, PC, 32, 1, 0), TCU_ERR_SHAPE);
    expect("poly overlap", tcu_poly_eval_ex(PA, 10, PB, 10, (void *)PB, 32, 1, 0),
           TCU_ERR_OVERLAP);
    expect("tc ld<n", tcu_transitive_closure_ex(PC, 100, 99, 32, 0), TCU_ERR_SHAPE);
    expect("tc huge", tcu_transitive_closure_ex(PC, 1 << 30, (int64_t)1 << 39, 32, 0),
           TCU_ERR_SHAPE);
    expect("tc empty", tcu_transitive_closure_ex(0, 0, 0, 32, 0), TCU_OK);
    expect("dft n", tcu_dft_ex(PA, PC, (void *)PB, 1000, 1, 32, 0), TCU_ERR_SHAPE);
    expect("dft batch huge", tcu_dft_ex(PA, PC, (void *)PB, 1 << 20, big, 32, 0), TCU_ERR_SHAPE);
    expect("dft work", tcu_dft_ex(PA, PC, 0, 1 << 20, 2, 32, 0), TCU_ERR_NULL);
    expect("dft valid", tcu_dft_ex(PA, PC, (void *)PB, 1 << 10, 2, 32, 0), TCU_ERR_NO_DEVICE);

    /* pointer check and strings */
    expect("range neg", tcu_check_device_range(PA, -1), TCU_ERR_SHAPE);
    expect("range empty", tcu_check_device_range(PA, 0), TCU_OK);
    for (int st = 1; st >= -9; --st)
        if (!tcu_strerror(st)) ++failures;

    expect("calls", (int)tcu_calls(), 0);
    printf("abi driver: %d failures\n", failures);
    return failures ? 1 : 0;
}
