"""GPU parity of the native tensor-unit call (Section 3, model definition:
C = A (n x s) * B (s x s)) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import compare, mm
from paper_1908_06649_amd import inputs, tcu

from gpu_util import DEV, draw_pair, run_tall, to_np

pytestmark = pytest.mark.gpu

DTYPES = [("f16", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("i8", "i32")]


def test_workload_f16_n4096_s16():
    spec = inputs.WORKLOADS["tall_f16_n4096_s16"]
    A, B = inputs.make_inputs(spec)
    got = run_tall(A, B, 16, "f32")
    rep = compare.check("f16", "f32", inputs.bits(A), inputs.bits(B), got)
    print(rep)


@pytest.mark.parametrize("din,dout", DTYPES)
@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("extra", [0, 1, 3, 17, 1000, 4099, 70001])
def test_dtypes_and_ragged_rows(din, dout, s, extra):
    n = s + extra                      # n >= s, mostly not a multiple of 16
    A, B = draw_pair((n, s), (s, s), din, seed=1000 * s + extra)
    got = run_tall(A, B, s, dout)
    compare.check(din, dout, inputs.bits(A), inputs.bits(B), got)


@pytest.mark.parametrize("din,dout", DTYPES)
@pytest.mark.parametrize("s", [16, 32])
def test_identity_weights(din, dout, s):
    n = 5 * s + 7
    A, _ = draw_pair((n, s), (s, s), din, seed=5)
    got = run_tall(A, inputs.identity(s, din), s, dout)
    want = A.to(inputs.TORCH_DTYPE[dout])
    assert np.array_equal(got, to_np(want))


@pytest.mark.parametrize("din,dout", DTYPES)
def test_permutation_weights(din, dout):
    s, n = 32, 333
    A, _ = draw_pair((n, s), (s, s), din, seed=6)
    P, perm = inputs.permutation(s, din, 7)
    got = run_tall(A, P, s, dout)
    want = A[:, perm].to(inputs.TORCH_DTYPE[dout])
    assert np.array_equal(got, to_np(want))


@pytest.mark.parametrize("din,dout", DTYPES)
@pytest.mark.parametrize("s", [16, 32])
def test_small_integers_bit_exact(din, dout, s):
    """Values in {-2..2}: every partial sum is an integer of magnitude <= 4s,
    exact in binary32 and in bfloat16, so the result is unique."""
    n = 4 * s + 9
    A = inputs.small_ints((n, s), din, 8)
    B = inputs.small_ints((s, s), din, 9)
    got = run_tall(A, B, s, dout)
    ref = mm(inputs.bits(A), inputs.bits(B), din)
    if dout == "bf16":       # integers of magnitude <= 128 are exact bfloat16 values
        got = compare.bf16_to_f64(got)
    assert np.array_equal(np.asarray(got, dtype=np.float64), np.asarray(ref, dtype=np.float64))


@pytest.mark.parametrize("din,dout", [("i8", "i32"), ("bf16", "bf16"), ("f16", "f32")])
@pytest.mark.parametrize("s", [16, 32])
def test_weak_model_stacked_square_calls(din, dout, s):
    """Section 5: an n x s call equals n/s stacked s x s calls."""
    n = 12 * s
    A, B = draw_pair((n, s), (s, s), din, seed=10)
    tall = run_tall(A, B, s, dout)
    stacked = np.concatenate([run_tall(A[q * s:(q + 1) * s].contiguous(), B, s, dout)
                              for q in range(n // s)])
    assert np.array_equal(tall, stacked)


def test_counts_one_call_per_invocation():
    s, n = 32, 1000
    A, B = draw_pair((n, s), (s, s), "bf16", seed=11)
    tcu.tcu_reset_calls()
    run_tall(A, B, s, "f32")
    assert tcu.tcu_calls() == 1
    assert tcu.tcu_square_calls() == (n + s - 1) // s
    assert tcu.tcu_work() == n * s


def test_rejected_call_leaves_output_untouched():
    s, n = 16, 64
    A = torch.zeros(n, s, dtype=torch.float16, device=DEV)
    B = torch.zeros(s, s, dtype=torch.float16, device=DEV)
    C = torch.full((n, s), 7.0, dtype=torch.float32, device=DEV)
    tcu.tcu_reset_calls()
    L = tcu.lib()
    # C overlapping A
    rc = L.tcu_mm_tall_ex(A.data_ptr(), n, s, B.data_ptr(), A.data_ptr(), tcu.TCU_F16_F32, None)
    assert rc == tcu.TCU_ERR_OVERLAP
    # misaligned A
    rc = L.tcu_mm_tall_ex(A.data_ptr() + 2, n - 1, s, B.data_ptr(), C.data_ptr(), 0, None)
    assert rc == tcu.TCU_ERR_ALIGN
    torch.cuda.synchronize()
    assert bool((C == 7.0).all()) and tcu.tcu_calls() == 0


def test_deterministic():
    s, n = 32, 50000
    A, B = draw_pair((n, s), (s, s), "bf16", seed=12)
    a = run_tall(A, B, s, "bf16")
    b = run_tall(A, B, s, "bf16")
    assert np.array_equal(a, b)


def test_workload_bf16_n16777216_s32_all_rows():
    """The very tall bf16 call at full size (2^24 x 32), every row against the
    oracle, in chunks of 2^20 rows (bf16 output: Frobenius against the
    oracle rounded once, elementwise and rounding-consistency bounds)."""
    spec = inputs.WORKLOADS["tall_bf16_n16777216_s32"]
    A, B = inputs.make_inputs(spec)
    n, s = spec["n"], spec["s"]
    got = run_tall(A, B, s, "bf16", check_guard=True)
    a_bits, b_bits = inputs.bits(A), inputs.bits(B)
    chunk = 1 << 20
    worst = 0.0
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        rep = compare.check("bf16", "bf16", a_bits[r0:r1], b_bits, got[r0:r1])
        worst = max(worst, rep["rel_frob_vs_rounded"])
    print("rows", n, "worst chunk rel_frob_vs_rounded", worst)
