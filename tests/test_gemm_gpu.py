"""GPU parity of the blocked dense multiplication of Theorem 2 (Section 4.1)
against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import compare, mm
from paper_1908_06649_amd import inputs, tcu

from gpu_util import DEV, PATHS, draw_pair, run_gemm, run_tall, to_np

pytestmark = pytest.mark.gpu

DTYPES = [("f16", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("i8", "i32")]


def test_workload_f16_N1024_s16():
    spec = inputs.WORKLOADS["gemm_f16_N1024_s16"]
    A, B = inputs.make_inputs(spec)
    got = run_gemm(A, B, 16, "f32")
    rep = compare.check("f16", "f32", inputs.bits(A), inputs.bits(B), got)
    print(rep)


# sizes spanning 1, several and ragged tiles (N is always a multiple of s)
SIZES = [(16, 16), (32, 16), (48, 16), (32, 32), (64, 32), (96, 32), (272, 16),
         (400, 16), (544, 32), (1056, 32), (2080, 32)]


@pytest.mark.parametrize("din,dout", DTYPES)
@pytest.mark.parametrize("N,s", SIZES)
def test_sizes_and_dtypes(din, dout, N, s):
    A, B = draw_pair((N, N), (N, N), din, seed=N * 7 + s)
    got = run_gemm(A, B, s, dout)
    compare.check(din, dout, inputs.bits(A), inputs.bits(B), got)


@pytest.mark.parametrize("N", [4352])
@pytest.mark.parametrize("din,dout", [("bf16", "f32"), ("i8", "i32")])
def test_big_tile_path_ragged(din, dout, N):
    """N above the big-tile threshold and not a multiple of the 256 tile."""
    A, B = draw_pair((N, N), (N, N), din, seed=N)
    got = run_gemm(A, B, 32, dout)
    rows = np.array([0, 1, 255, 256, 1000, 4095, 4096, 4351])
    compare.check(din, dout, inputs.bits(A), inputs.bits(B), got[rows], rows=rows)


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("N", [96, 128])
def test_composition_of_tall_calls(N, s):
    """Theorem 2: tcu_gemm equals sum_i A_i * B_{i,j} computed with one native
    call per (i, j) and summed on the host -- bit-exact for int8."""
    A, B = draw_pair((N, N), (N, N), "i8", seed=N + s)
    full = run_gemm(A, B, s, "i32").astype(np.int64)
    q = N // s
    acc = np.zeros((N, N), dtype=np.int64)
    tcu.tcu_reset_calls()
    for i in range(q):
        Ai = A[:, i * s:(i + 1) * s].contiguous()
        for j in range(q):
            Bij = B[i * s:(i + 1) * s, j * s:(j + 1) * s].contiguous()
            acc[:, j * s:(j + 1) * s] += run_tall(Ai, Bij, s, "i32").astype(np.int64)
    assert tcu.tcu_calls() == q * q
    assert np.array_equal(full, acc)


@pytest.mark.parametrize("din,dout", DTYPES)
def test_identity_and_permutation(din, dout):
    N, s = 512, 32
    A, _ = draw_pair((N, N), (N, N), din, seed=3)
    got = run_gemm(A, inputs.identity(N, din), s, dout)
    assert np.array_equal(got, to_np(A.to(inputs.TORCH_DTYPE[dout])))
    P, perm = inputs.permutation(N, din, 4)
    got = run_gemm(A, P, s, dout)
    assert np.array_equal(got, to_np(A[:, perm].to(inputs.TORCH_DTYPE[dout])))


@pytest.mark.parametrize("din", ["f16", "bf16", "i8"])
def test_small_integers_bit_exact(din):
    """Values in {-2..2}: sums are integers of magnitude <= 4N, exact in binary32."""
    N, s = 800, 16
    A = inputs.small_ints((N, N), din, 5)
    B = inputs.small_ints((N, N), din, 6)
    got = run_gemm(A, B, s, "i32" if din == "i8" else "f32")
    ref = mm(inputs.bits(A), inputs.bits(B), din)
    assert np.array_equal(np.asarray(got, dtype=np.float64), np.asarray(ref, dtype=np.float64))


def test_counts_calls_of_theorem_2():
    N, s = 256, 32
    A, B = draw_pair((N, N), (N, N), "bf16", seed=9)
    tcu.tcu_reset_calls()
    run_gemm(A, B, s, "f32")
    q = N // s
    assert tcu.tcu_calls() == q * q               # n/m calls, n = N^2, m = s^2
    assert tcu.tcu_square_calls() == q ** 3
    assert tcu.tcu_work() == N ** 3 // s          # N^3 / sqrt(m) model work


def test_int8_deterministic():
    N = 1024
    A, B = draw_pair((N, N), (N, N), "i8", seed=10)
    assert np.array_equal(run_gemm(A, B, 32, "i32"), run_gemm(A, B, 32, "i32"))


def test_workload_bf16_N8192_s32_all_rows():
    """The headline product at full size, every element against the binary64
    oracle (relative Frobenius and elementwise bounds)."""
    spec = inputs.WORKLOADS["gemm_bf16_N8192_s32"]
    A, B = inputs.make_inputs(spec)
    got = run_gemm(A, B, 32, "f32")
    rep = compare.check("bf16", "f32", inputs.bits(A), inputs.bits(B), got)
    print(rep)


def test_workload_i8_N8192_s32_all_rows():
    """The int8 product at full size, bit-exact on all 8192 x 8192 elements
    (the product of Theorem 2 is unique in int32 here)."""
    spec = inputs.WORKLOADS["gemm_i8_N8192_s32"]
    A, B = inputs.make_inputs(spec)
    got = run_gemm(A, B, 32, "i32")
    rep = compare.check("i8", "i32", inputs.bits(A), inputs.bits(B), got)
    assert rep["mismatches"] == 0


# Every kernel of the product on sizes where it applies (N % 256 == 0): the
# full-tile kernel (DMA-fed LDS ring, transposing reads), the general one
# (register-staged, predicated tails) and the small-tile ring kernel (16-bit
# inputs; int8 falls back to the general kernel under "ring").
@pytest.mark.parametrize("path", ["fast", "general", "ring"])
@pytest.mark.parametrize("din,dout", DTYPES)
@pytest.mark.parametrize("N,s", [(256, 16), (512, 32), (1280, 32)])
def test_kernel_paths(knobs, path, din, dout, N, s):
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, PATHS[path])
    A, B = draw_pair((N, N), (N, N), din, seed=N + 3 * s)
    got = run_gemm(A, B, s, dout)
    compare.check(din, dout, inputs.bits(A), inputs.bits(B), got)


@pytest.mark.parametrize("path", ["fast", "general", "ring"])
@pytest.mark.parametrize("din,dout", DTYPES)
def test_kernel_paths_identity_permutation(knobs, path, din, dout):
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, PATHS[path])
    N, s = 768, 16
    A, _ = draw_pair((N, N), (N, N), din, seed=11)
    got = run_gemm(A, inputs.identity(N, din), s, dout)
    assert np.array_equal(got, to_np(A.to(inputs.TORCH_DTYPE[dout])))
    P, perm = inputs.permutation(N, din, 12)
    got = run_gemm(A, P, s, dout)
    assert np.array_equal(got, to_np(A[:, perm].to(inputs.TORCH_DTYPE[dout])))


@pytest.mark.parametrize("path", ["fast", "general"])
def test_kernel_paths_composition(knobs, path):
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, PATHS[path])
    N, s = 256, 32
    A, B = draw_pair((N, N), (N, N), "i8", seed=13)
    full = run_gemm(A, B, s, "i32").astype(np.int64)
    q = N // s
    acc = np.zeros((N, N), dtype=np.int64)
    for i in range(q):
        Ai = A[:, i * s:(i + 1) * s].contiguous()
        for j in range(q):
            Bij = B[i * s:(i + 1) * s, j * s:(j + 1) * s].contiguous()
            acc[:, j * s:(j + 1) * s] += run_tall(Ai, Bij, s, "i32").astype(np.int64)
    assert np.array_equal(full, acc)
