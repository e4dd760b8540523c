"""C ABI tests that need no GPU: the library loads, exports every function
include/tcu.h declares, and rejects bad arguments before any HIP call.

Every call below with non-NULL fake pointers is built to fail validation, so
no kernel can ever be launched on them.  The one call with valid arguments
(expecting TCU_ERR_NO_DEVICE) runs only where no GPU is visible.
"""
import os
import re
import subprocess
import threading

import pytest
import torch

from paper_1908_06649_amd import tcu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tcu.h")

# fake, 16-byte aligned, far-apart "device" addresses (never dereferenced)
PA, PB, PC = 0x10000000, 0x20000000, 0x30000000


@pytest.fixture(scope="module")
def L():
    lib = tcu.lib()
    lib.tcu_set_unit(16)
    lib.tcu_set_dtype(tcu.TCU_F16_F32)
    lib.tcu_reset_calls()
    return lib


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tcu_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("tcu_mm_tall", "tcu_gemm", "tcu_set_unit", "tcu_set_dtype",
                 "tcu_set_stream", "tcu_calls", "tcu_reset_calls", "tcu_strerror"):
        assert must in names


def test_library_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(tcu.SIGNATURES), "binding and header disagree"
    out = subprocess.run(["nm", "-D", "--defined-only", tcu.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (tcu_[a-z0-9_]+)$", out, flags=re.M))
    assert set(names) <= exported
    for n in names:
        assert getattr(L, n) is not None


def test_strerror_covers_all_codes(L):
    for code in range(0, -10, -1):
        msg = tcu.tcu_strerror(code)
        assert msg and "unknown" not in msg
    assert "unknown" in tcu.tcu_strerror(-99)


def test_unit_and_dtype_config(L):
    assert L.tcu_set_unit(32) == tcu.TCU_OK and L.tcu_get_unit() == 32
    assert L.tcu_set_unit(8) == tcu.TCU_ERR_UNSUPPORTED and L.tcu_get_unit() == 32
    assert L.tcu_set_unit(64) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_unit(16) == tcu.TCU_OK
    assert L.tcu_set_dtype(tcu.TCU_I8_I32) == tcu.TCU_OK and L.tcu_get_dtype() == tcu.TCU_I8_I32
    assert L.tcu_set_dtype(4) == tcu.TCU_ERR_UNSUPPORTED and L.tcu_get_dtype() == tcu.TCU_I8_I32
    assert L.tcu_set_dtype(-1) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_dtype(tcu.TCU_F16_F32) == tcu.TCU_OK
    assert L.tcu_set_stream(0x1234) == tcu.TCU_OK and L.tcu_get_stream() == 0x1234
    assert L.tcu_set_stream(None) == tcu.TCU_OK and not L.tcu_get_stream()


def test_knobs_set_get_and_reject(L):
    """Test overrides: set, read back, reset; unknown knobs and values out of
    range are rejected and leave the knob unchanged."""
    for knob, good in ((tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_RING), (tcu.TCU_KNOB_PP_GRID, 3),
                       (tcu.TCU_KNOB_SPLIT_K, 4), (tcu.TCU_KNOB_TAIL_SPLIT, 1),
                       (tcu.TCU_KNOB_CHECK_POINTERS, 1), (tcu.TCU_KNOB_DFT_PAIRS, 1)):
        start = L.tcu_get_knob(knob)
        assert L.tcu_set_knob(knob, good) == tcu.TCU_OK and L.tcu_get_knob(knob) == good
        assert L.tcu_set_knob(knob, -1) == tcu.TCU_ERR_UNSUPPORTED
        assert L.tcu_get_knob(knob) == good
        assert L.tcu_set_knob(knob, start) == tcu.TCU_OK
    assert L.tcu_set_knob(tcu.TCU_KNOB_GEMM_KERNEL, 4) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_knob(tcu.TCU_KNOB_CHECK_POINTERS, 2) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_knob(tcu.TCU_KNOB_DFT_PAIRS, 2) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_knob(6, 0) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_set_knob(-1, 0) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_get_knob(6) == -1 and L.tcu_get_knob(-1) == -1


def test_debug_env_turns_pointer_checks_on():
    """TCU_DEBUG at load time sets the initial pointer-check knob (a fresh
    process, since the environment is read once when the library loads)."""
    code = ("from paper_1908_06649_amd import tcu; "
            "print(tcu.tcu_get_knob(tcu.TCU_KNOB_CHECK_POINTERS))")
    for env_val, want in (("1", "1"), ("0", "0"), (None, "0")):
        env = dict(os.environ)
        env.pop("TCU_DEBUG", None)
        if env_val is not None:
            env["TCU_DEBUG"] = env_val
        out = subprocess.run([os.sys.executable, "-c", code], cwd=ROOT, env=env,
                             capture_output=True, text=True, check=True).stdout.strip()
        assert out.splitlines()[-1] == want, (env_val, out)


def test_check_device_range_arguments(L):
    assert L.tcu_check_device_range(PA, 0) == tcu.TCU_OK        # empty range: nothing to check
    assert L.tcu_check_device_range(PA, -1) == tcu.TCU_ERR_SHAPE
    if not torch.cuda.is_available():
        assert L.tcu_check_device_range(PA, 16) == tcu.TCU_ERR_NO_DEVICE


def test_config_is_per_thread(L):
    L.tcu_set_unit(16)
    seen = {}

    def worker():
        seen["before"] = L.tcu_get_unit()
        L.tcu_set_unit(32)
        seen["after"] = L.tcu_get_unit()

    t = threading.Thread(target=worker)
    t.start()
    t.join()
    assert seen == {"before": 16, "after": 32}
    assert L.tcu_get_unit() == 16


TALL_ERRORS = [
    # (A, n, s, B, C, dtype) -> status
    ((0, 4096, 16, PB, PC, 0), tcu.TCU_ERR_NULL),
    ((PA, 4096, 16, 0, PC, 0), tcu.TCU_ERR_NULL),
    ((PA, 4096, 16, PB, 0, 0), tcu.TCU_ERR_NULL),
    ((PA, 4096, 8, PB, PC, 0), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 4096, 24, PB, PC, 0), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 4096, 16, PB, PC, 4), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 4096, 16, PB, PC, -1), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 15, 16, PB, PC, 0), tcu.TCU_ERR_SHAPE),          # n < s
    ((PA, 31, 32, PB, PC, 1), tcu.TCU_ERR_SHAPE),
    ((PA, 0, 16, PB, PC, 0), tcu.TCU_ERR_SHAPE),
    ((PA, -5, 16, PB, PC, 0), tcu.TCU_ERR_SHAPE),
    ((PA, (1 << 40) + 1, 16, PB, PC, 0), tcu.TCU_ERR_SHAPE),
    ((PA + 8, 4096, 16, PB, PC, 0), tcu.TCU_ERR_ALIGN),
    ((PA, 4096, 16, PB + 2, PC, 0), tcu.TCU_ERR_ALIGN),
    ((PA, 4096, 16, PB, PC + 4, 0), tcu.TCU_ERR_ALIGN),
    # C overlaps A: A spans 4096*16*2 bytes
    ((PA, 4096, 16, PB, PA + 4096 * 16 * 2 - 16, 0), tcu.TCU_ERR_OVERLAP),
    ((PA, 4096, 16, PB, PA - 4096 * 16 * 4 + 16, 0), tcu.TCU_ERR_OVERLAP),
    # C overlaps B (B spans 16*16*2 bytes; C starts inside it)
    ((PA, 4096, 16, PB, PB + 496, 0), tcu.TCU_ERR_OVERLAP),
]


@pytest.mark.parametrize("args,want", TALL_ERRORS)
def test_tall_rejects(L, args, want):
    L.tcu_reset_calls()
    A, n, s, B, C, dt = args
    assert L.tcu_mm_tall_ex(A, n, s, B, C, dt, None) == want
    assert L.tcu_calls() == 0 and L.tcu_square_calls() == 0 and L.tcu_work() == 0


def test_tall_stateful_checks_unit(L):
    L.tcu_set_unit(16)
    assert L.tcu_mm_tall(PA, 4096, 32, PB, PC) == tcu.TCU_ERR_UNSUPPORTED
    assert L.tcu_mm_tall(0, 4096, 16, PB, PC) == tcu.TCU_ERR_NULL
    assert L.tcu_mm_tall(PA, 8, 16, PB, PC) == tcu.TCU_ERR_SHAPE


GEMM_ERRORS = [
    # (A, B, C, N, s, dtype) -> status
    ((0, PB, PC, 1024, 16, 0), tcu.TCU_ERR_NULL),
    ((PA, 0, PC, 1024, 16, 0), tcu.TCU_ERR_NULL),
    ((PA, PB, 0, 1024, 16, 0), tcu.TCU_ERR_NULL),
    ((PA, PB, PC, 1024, 12, 0), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, PB, PC, 1024, 16, 9), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, PB, PC, 1000, 16, 0), tcu.TCU_ERR_SHAPE),          # N % s != 0
    ((PA, PB, PC, 48, 32, 1), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, 16, 32, 1), tcu.TCU_ERR_SHAPE),            # N < s
    ((PA, PB, PC, 0, 16, 0), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, (1 << 20) + 16, 16, 0), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, 1 << 17, 32, 3), tcu.TCU_ERR_SHAPE),       # int32 sums could overflow
    ((PA + 4, PB, PC, 1024, 16, 0), tcu.TCU_ERR_ALIGN),
    ((PA, PB, PC + 8, 1024, 16, 0), tcu.TCU_ERR_ALIGN),
    ((PA, PB, PA + 1024 * 1024 * 2 - 16, 1024, 16, 0), tcu.TCU_ERR_OVERLAP),
    ((PA, PB, PB, 1024, 16, 0), tcu.TCU_ERR_OVERLAP),
]


@pytest.mark.parametrize("args,want", GEMM_ERRORS)
def test_gemm_rejects(L, args, want):
    L.tcu_reset_calls()
    A, B, C, N, s, dt = args
    assert L.tcu_gemm_ex(A, B, C, N, s, dt, None) == want
    assert L.tcu_calls() == 0


def test_gemm_stateful_uses_unit(L):
    L.tcu_set_unit(32)
    L.tcu_set_dtype(tcu.TCU_BF16_F32)
    assert L.tcu_gemm(PA, PB, PC, 48) == tcu.TCU_ERR_SHAPE     # 48 % 32 != 0
    L.tcu_set_unit(16)
    L.tcu_set_dtype(tcu.TCU_F16_F32)


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a HIP device is visible")
def test_valid_arguments_without_device(L):
    L.tcu_reset_calls()
    assert L.tcu_mm_tall_ex(PA, 4096, 16, PB, PC, 0, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_gemm_ex(PA, PB, PC, 1024, 16, 0, None) == tcu.TCU_ERR_NO_DEVICE
    # A and B may overlap (both are only read)
    assert L.tcu_gemm_ex(PA, PA, PC, 1024, 16, 0, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_calls() == 0


def test_python_binding_marshalling_errors():
    A = torch.zeros(64, 16, dtype=torch.float16)
    B = torch.zeros(16, 16, dtype=torch.float16)
    C = torch.zeros(64, 16, dtype=torch.float32)
    with pytest.raises(ValueError):          # host tensors are not device memory
        tcu.tcu_mm_tall(A, 64, 16, B, C)
    with pytest.raises(tcu.TcuError):        # unsupported dtype pair
        tcu.tcu_mm_tall(A, 64, 16, B, C.to(torch.float16))


# ------------------------------------------------ rectangular / accumulate
NO_DEV = torch.cuda.device_count() == 0

RECT_ERRORS = [
    # (A, lda, B, ldb, C, ldc, M, K, N, flags, s, dtype) -> status
    ((0, 64, PB, 64, PC, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_NULL),
    ((PA, 64, PB, 64, 0, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_NULL),
    ((PA, 64, PB, 64, PC, 64, 64, 64, 64, 2, 16, 0), tcu.TCU_ERR_UNSUPPORTED),   # unknown flag
    ((PA, 64, PB, 64, PC, 64, 64, 64, 64, 0, 8, 0), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 64, PB, 64, PC, 64, 64, 64, 64, 0, 16, 7), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 64, PB, 64, PC, 64, -1, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),
    ((PA, 64, PB, 64, PC, 64, 64, -1, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),
    ((PA, 1 << 31, PB, 64, PC, 64, 2, (1 << 30) + 1, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),
    ((PA, 1 << 17, PB, 64, PC, 64, 64, 1 << 17, 64, 0, 32, 3), tcu.TCU_ERR_SHAPE),  # int8 K
    ((PA, 63, PB, 64, PC, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),        # lda < K
    ((PA, 64, PB, 63, PC, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),        # ldb < N
    ((PA, 64, PB, 64, PC, 63, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),        # ldc < N
    ((PA, 1 << 40, PB, 64, PC, 64, 2, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),    # pitch too big
    ((PA, 1 << 30, PB, 64, PC, 64, 1024, 64, 64, 0, 16, 0), tcu.TCU_ERR_SHAPE),  # extent 2^41 B
    ((PA + 2, 64, PB, 64, PC, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_ALIGN),
    ((PA, 64, PB, 64, PC + 8, 64, 64, 64, 64, 0, 16, 0), tcu.TCU_ERR_ALIGN),
    # C is A (same block)
    ((PA, 64, PB, 64, PA, 64, 64, 64, 64, 0, 16, 2), tcu.TCU_ERR_OVERLAP),
    # C = columns 32..95 of a 1024-wide bf16 array, A = columns 0..63: shared columns
    ((PA, 1024, PB, 64, PA + 64, 1024, 64, 64, 64, 0, 16, 2), tcu.TCU_ERR_OVERLAP),
    # C's rows start 64 bytes before the end of A's grid rows and wrap into row 1
    ((PA, 1024, PB, 64, PA + 2048 - 64, 1024, 64, 64, 64, 0, 16, 2), tcu.TCU_ERR_OVERLAP),
    # different byte pitches over the same range: reported conservatively
    ((PA, 1024, PB, 64, PA + 1024, 512, 64, 64, 64, 0, 16, 2), tcu.TCU_ERR_OVERLAP),
    # C overlaps B
    ((PA, 64, PB, 64, PB + 64 * 128 - 16, 64, 64, 64, 64, 1, 16, 2), tcu.TCU_ERR_OVERLAP),
]


# Extents whose int64 product would wrap around: the validation (128-bit,
# saturating) must see them as too large, not as small or negative sizes.
# (Run only where no device is visible: a wrong acceptance must not reach a
# launch.)
RECT_OVERFLOW = [
    (PA, 1 << 39, PB, 64, PC, 64, 1 << 30, 1, 64, 0, 16, 0),      # (M-1) lda ~ 2^69
    (PA, 64, PB, 1 << 39, PC, 64, 64, 1 << 30, 64, 0, 16, 0),     # (K-1) ldb
    (PA, 64, PB, 64, PC, (1 << 40) - 16, 1 << 30, 64, 64, 0, 16, 0),  # (M-1) ldc * 4
]


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a HIP device is visible")
@pytest.mark.parametrize("args", RECT_OVERFLOW)
def test_rect_rejects_wrapping_extents(L, args):
    L.tcu_reset_calls()
    assert L.tcu_gemm_rect_ex(*args, None) == tcu.TCU_ERR_SHAPE
    assert L.tcu_calls() == 0


@pytest.mark.parametrize("args,want", RECT_ERRORS)
def test_rect_rejects(L, args, want):
    L.tcu_reset_calls()
    assert L.tcu_gemm_rect_ex(*args, None) == want
    assert L.tcu_calls() == 0 and L.tcu_work() == 0


def test_rect_empty_is_a_noop(L):
    """M = 0, N = 0, or K = 0 when accumulating: success with no device work
    and no calls (fake pointers are never touched)."""
    L.tcu_reset_calls()
    assert L.tcu_gemm_rect_ex(PA, 64, PB, 64, PC, 64, 0, 64, 64, 0, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_gemm_rect_ex(PA, 64, PB, 64, PC, 64, 64, 64, 0, 1, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_gemm_rect_ex(PA, 64, PB, 64, PC, 64, 64, 0, 64, 1, 32, 3, None) == tcu.TCU_OK
    # operands without elements may be NULL
    assert L.tcu_gemm_rect_ex(None, 0, None, 64, PC, 64, 64, 0, 64, 1, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_gemm_rect_ex(None, 64, PB, 64, None, 64, 0, 64, 64, 0, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_gemm_rect_ex(PA, 64, None, 0, None, 0, 64, 64, 0, 0, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_gemm_rect_ex(None, 0, None, 64, None, 64, 64, 0, 64, 1, 16, 0, None) \
        == tcu.TCU_ERR_NULL
    assert L.tcu_calls() == 0 and L.tcu_square_calls() == 0 and L.tcu_work() == 0


@pytest.mark.skipif(not NO_DEV, reason="a HIP device is visible (valid calls would launch)")
def test_rect_disjoint_blocks_of_one_array_pass(L):
    """The D functions update one block of an array from two others: with one
    byte pitch the check is element-exact, so disjoint blocks are accepted."""
    P = 1024 * 2      # bytes per row of a 1024-wide bfloat16 array at PA
    blk = lambda r, c: PA + r * P + c * 2
    # X = block (0, 64), Y = block (0, 0), Z = block (64, 64), all 64 x 64
    rc = L.tcu_gemm_rect_ex(blk(0, 0), 1024, blk(64, 64), 1024, blk(0, 64), 1024,
                            64, 64, 64, tcu.TCU_ACCUMULATE, 16, tcu.TCU_BF16_BF16, None)
    assert rc == tcu.TCU_ERR_NO_DEVICE
    # X right next to Y in the same rows, and X = the block just below Y
    assert L.tcu_gemm_rect_ex(blk(0, 0), 1024, blk(64, 0), 1024, blk(0, 64), 1024,
                              64, 64, 64, 1, 16, 2, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_gemm_rect_ex(blk(0, 0), 1024, blk(0, 64), 1024, blk(64, 0), 1024,
                              64, 64, 64, 1, 16, 2, None) == tcu.TCU_ERR_NO_DEVICE


def _brute_overlap(a, ar, aw, ap, b, br, bw, bp):
    """Do two row-major byte views share a byte?  (set intersection)"""
    sa = {a + i * ap + j for i in range(ar) for j in range(aw)}
    return any(b + i * bp + j in sa for i in range(br) for j in range(bw))


@pytest.mark.skipif(not NO_DEV, reason="a HIP device is visible (valid calls would launch)")
def test_rect_overlap_check_vs_brute_force(L):
    """The element-exact overlap test against set intersection on small
    random views of one bfloat16 array (2-byte elements in and out): exact
    when the pitches agree, never missing a real overlap otherwise."""
    import random
    rng = random.Random(5)
    n_same = n_hit = 0
    for _ in range(3000):
        M, K, N = rng.randint(1, 4), rng.randint(1, 24), rng.randint(1, 24)
        lda = K + 8 * rng.randint(0, 3)
        ldc = lda if rng.random() < 0.7 else N + 8 * rng.randint(0, 3)
        ldc = max(ldc, N)
        offa = 16 * rng.randint(0, 40)
        offc = 16 * rng.randint(0, 40)
        A, C = PA + offa, PA + offc
        rc = L.tcu_gemm_rect_ex(A, lda, PB, N, C, ldc, M, K, N, 0, 16, tcu.TCU_BF16_BF16, None)
        real = _brute_overlap(C, M, 2 * N, 2 * ldc, A, M, 2 * K, 2 * lda)
        if real:
            n_hit += 1
            assert rc == tcu.TCU_ERR_OVERLAP
        same_pitch = ldc == lda or M == 1
        if same_pitch and not real:
            assert rc == tcu.TCU_ERR_NO_DEVICE, (M, K, N, lda, ldc, offa, offc)
        if same_pitch:
            n_same += 1
    assert n_same > 1000 and n_hit > 300


def test_python_rect_marshalling_errors():
    A = torch.zeros(64, 32, dtype=torch.bfloat16)
    B = torch.zeros(32, 16, dtype=torch.bfloat16)
    C = torch.zeros(64, 16, dtype=torch.float32)
    with pytest.raises(ValueError):          # host tensors
        tcu.tcu_gemm_rect(A, 32, B, 16, C, 16, 64, 32, 16)


# ---- polynomial evaluation, transitive closure, DFT: argument checks ----

POLY_ERRORS = [
    # (coef, n, points, p, out, s, dtype) -> status
    ((PA, 100, PB, 64, PC, 8, 1), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, 100, PB, 64, PC, 32, 3), tcu.TCU_ERR_UNSUPPORTED),     # int8 has no polynomial form
    ((PA, 100, PB, 64, PC, 32, 9), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, -1, PB, 64, PC, 32, 1), tcu.TCU_ERR_SHAPE),
    ((PA, 100, PB, -1, PC, 32, 1), tcu.TCU_ERR_SHAPE),
    ((PA, (1 << 40) + 1, PB, 64, PC, 32, 1), tcu.TCU_ERR_SHAPE),
    ((PA, 100, PB, (1 << 40) + 1, PC, 32, 1), tcu.TCU_ERR_SHAPE),
    ((0, 100, PB, 64, PC, 32, 1), tcu.TCU_ERR_NULL),
    ((PA, 100, 0, 64, PC, 32, 1), tcu.TCU_ERR_NULL),
    ((PA, 100, PB, 64, 0, 32, 1), tcu.TCU_ERR_NULL),
    ((PA + 8, 100, PB, 64, PC, 32, 1), tcu.TCU_ERR_ALIGN),
    ((PA, 100, PB, 64, PC + 4, 32, 1), tcu.TCU_ERR_ALIGN),
    ((PA, 100, PB, 64, PB + 64, 32, 1), tcu.TCU_ERR_OVERLAP),      # out over the points
    ((PA, 100, PB, 64, PA + 192, 32, 0), tcu.TCU_ERR_OVERLAP),     # out over the coefficients
]


@pytest.mark.parametrize("args,want", POLY_ERRORS)
def test_poly_rejects(L, args, want):
    L.tcu_reset_calls()
    assert L.tcu_poly_eval_ex(*args, None) == want
    assert L.tcu_calls() == 0


def test_poly_empty_needs_no_device(L):
    """p = 0 (nothing to evaluate) succeeds before any device call; NULL
    arrays are allowed when empty."""
    L.tcu_reset_calls()
    assert L.tcu_poly_eval_ex(PA, 100, 0, 0, 0, 32, 1, None) == tcu.TCU_OK
    assert L.tcu_poly_eval_ex(0, 0, 0, 0, 0, 16, 0, None) == tcu.TCU_OK
    assert L.tcu_calls() == 0


TC_ERRORS = [
    # (X, n, ld, s) -> status
    ((PA, 64, 64, 8), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, -1, 64, 32), tcu.TCU_ERR_SHAPE),
    ((PA, (1 << 30) + 1, (1 << 30) + 1, 32), tcu.TCU_ERR_SHAPE),
    ((PA, 64, 63, 32), tcu.TCU_ERR_SHAPE),                         # ld < n
    ((PA, 1 << 20, 1 << 21, 32), tcu.TCU_ERR_SHAPE),               # extent 2^41 bytes
    ((0, 64, 64, 32), tcu.TCU_ERR_NULL),
    ((PA + 4, 64, 64, 32), tcu.TCU_ERR_ALIGN),
]


@pytest.mark.parametrize("args,want", TC_ERRORS)
def test_tc_rejects(L, args, want):
    L.tcu_reset_calls()
    assert L.tcu_transitive_closure_ex(*args, None) == want
    assert L.tcu_calls() == 0


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a HIP device is visible")
def test_tc_rejects_wrapping_extent(L):
    """(n - 1) ld ~ 2^82 must read as too large, not wrap around."""
    assert L.tcu_transitive_closure_ex(PA, 1 << 20, 1 << 62, 32, None) == tcu.TCU_ERR_SHAPE


def test_tc_empty_needs_no_device(L):
    L.tcu_reset_calls()
    assert L.tcu_transitive_closure_ex(0, 0, 0, 32, None) == tcu.TCU_OK
    assert L.tcu_calls() == 0


DFT_ERRORS = [
    # (x, y, work, n, batch, s) -> status
    ((PA, PB, PC, 1024, 1, 8), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, PB, PC, 0, 1, 32), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, 96, 1, 32), tcu.TCU_ERR_SHAPE),                  # not a power of two
    ((PA, PB, PC, (1 << 30) * 2, 1, 32), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, 1024, -1, 32), tcu.TCU_ERR_SHAPE),
    ((PA, PB, PC, 1 << 30, 1 << 7, 32), tcu.TCU_ERR_SHAPE),        # 2^40 bytes
    ((0, PB, PC, 1024, 1, 32), tcu.TCU_ERR_NULL),
    ((PA, 0, PC, 1024, 1, 32), tcu.TCU_ERR_NULL),
    ((PA, PB, 0, 1024, 1, 32), tcu.TCU_ERR_NULL),                  # two levels need work
    ((PA + 8, PB, PC, 1024, 1, 32), tcu.TCU_ERR_ALIGN),
    ((PA, PB, PC + 8, 1024, 1, 32), tcu.TCU_ERR_ALIGN),
    ((PA, PA + 4096, PC, 1024, 1, 32), tcu.TCU_ERR_OVERLAP),       # y over x
    ((PA, PB, PB + 8192 - 16, 1024, 1, 32), tcu.TCU_ERR_OVERLAP),  # work over y
    ((PA, PB, PA, 1024, 1, 32), tcu.TCU_ERR_OVERLAP),              # work over x
]


@pytest.mark.parametrize("args,want", DFT_ERRORS)
def test_dft_rejects(L, args, want):
    L.tcu_reset_calls()
    assert L.tcu_dft_ex(*args, None) == want
    assert L.tcu_calls() == 0


def test_dft_empty_batch_needs_no_device(L):
    L.tcu_reset_calls()
    assert L.tcu_dft_ex(0, 0, 0, 1024, 0, 32, None) == tcu.TCU_OK
    assert L.tcu_calls() == 0


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a HIP device is visible")
def test_new_entry_points_valid_arguments_without_device(L):
    """Valid arguments get as far as the device check (one level needs no
    work buffer)."""
    assert L.tcu_poly_eval_ex(PA, 100, PB, 64, PC, 32, 1, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_transitive_closure_ex(PA, 64, 64, 32, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_dft_ex(PA, PB, 0, 32, 4, 32, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_dft_ex(PA, PB, PC, 1 << 20, 4, 32, None) == tcu.TCU_ERR_NO_DEVICE


NOALLOC_ERRORS = [
    # (x, y, n, batch, s) -> status; the levels' second buffer is the library's
    ((PA, PB, 1024, 1, 8), tcu.TCU_ERR_UNSUPPORTED),
    ((PA, PB, 96, 1, 32), tcu.TCU_ERR_SHAPE),
    ((0, PB, 1024, 1, 32), tcu.TCU_ERR_NULL),
    ((PA, PB + 8, 1024, 1, 32), tcu.TCU_ERR_ALIGN),
    ((PA, PA + 4096, 1024, 1, 32), tcu.TCU_ERR_OVERLAP),
    # two levels: batch * n * 8 bytes above the fixed scratch
    ((PA, PC, 1 << 20, 9, 32), tcu.TCU_ERR_SCRATCH),
    ((PA, PC, 1 << 24, 1, 32), tcu.TCU_ERR_SCRATCH),
]


@pytest.mark.parametrize("args,want", NOALLOC_ERRORS)
def test_dft_noalloc_rejects(L, args, want):
    L.tcu_reset_calls()
    assert L.tcu_dft_noalloc(*args, None) == want
    assert L.tcu_calls() == 0


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a HIP device is visible")
def test_dft_noalloc_limits_without_device(L):
    """At the scratch limit, and a one-level transform of any size (no
    scratch needed), the call gets as far as the device check."""
    assert tcu.TCU_DFT_NOALLOC_MAX_BYTES == 64 << 20
    assert L.tcu_dft_noalloc(PA, 0x4000000000, 1 << 20, 8, 32, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_dft_noalloc(PA, 0x4000000000, 32, 1 << 24, 32, None) == tcu.TCU_ERR_NO_DEVICE
    assert L.tcu_dft_noalloc(0, 0, 1024, 0, 32, None) == tcu.TCU_OK
