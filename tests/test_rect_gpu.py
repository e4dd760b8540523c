"""GPU parity of the rectangular, strided and accumulating product
(tcu_gemm_rect: Corollary 1 through Theorem 2's strips and blocks, zero
padding of ragged dimensions, and the update X <- X + Y*Z of the D functions
of Sections 4.2 and 4.3) against the CPU oracle, through the C ABI.

Every case checks, besides the values, that the call wrote nothing outside
its M x N view of C, and the input arrays' unused columns hold NaN (int8:
127) so that a kernel reading past a view's K or N columns fails the
comparison.
"""
import numpy as np
import pytest
import torch

from oracle import compare
from paper_1908_06649_amd import inputs, tcu
import gpu_util as gu

pytestmark = pytest.mark.gpu

PAIRS = [("f16", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("i8", "i32")]
ES = {"f16": 2, "bf16": 2, "i8": 1}
OB = {"f32": 4, "bf16": 2, "i32": 4}


def aligned_pitch(cols: int, es: int, extra: int = 0) -> int:
    """Smallest pitch >= cols whose byte size is a multiple of 16, plus extra
    16-byte steps."""
    step = 16 // es
    return ((cols + step - 1) // step + extra) * step


def to_np_c0(C0: torch.Tensor, out: str) -> np.ndarray:
    if out == "bf16":
        return C0.view(torch.int16).numpy().view(np.uint16)
    return C0.numpy()


def run_and_check(M, K, N, din, out, s, pitch, accumulate, seed):
    A, B = gu.draw_pair((M, K), (K, N), din, seed)
    if pitch == "contiguous":
        lda, ldb, ldc = K, N, N
    else:
        lda = aligned_pitch(K, ES[din], 1)
        ldb = aligned_pitch(N, ES[din], 2)
        ldc = aligned_pitch(N, OB[out], 1)
    C0 = gu.c0_draw((M, N), out, seed + 1000) if accumulate else None
    got = gu.run_rect(A, B, s, din, out, lda, ldb, ldc, C0=C0)
    return compare.check(din, out, inputs.bits(A), inputs.bits(B), got,
                         C0=None if C0 is None else to_np_c0(C0, out))


# Ragged shapes: none, some or all dimensions multiples of the unit or of a
# tile; tiny, below one unit, and several tiles with tails.
RAGGED = [(1, 1, 1), (5, 7, 3), (16, 16, 16), (17, 33, 65), (64, 48, 80),
          (100, 130, 70), (255, 257, 129), (300, 1000, 260), (513, 77, 1030)]


@pytest.mark.parametrize("pitch", ["contiguous", "padded"])
@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("M,K,N", RAGGED)
def test_rect_ragged(M, K, N, din, out, accumulate, pitch):
    s = 32 if din == "bf16" else 16
    run_and_check(M, K, N, din, out, s, pitch, accumulate, seed=M * 7 + K * 3 + N)


# Whole 256 x 256 tiles and whole K stages: the full-tile kernel, forced, on
# rectangular shapes with padded pitches, against the general kernel.
FULL = [(256, 32, 256), (256, 64, 512), (512, 1024, 768), (768, 2048, 256)]


@pytest.mark.parametrize("kernel", ["fast", "general"])
@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("M,K,N", FULL)
def test_rect_full_tiles(M, K, N, din, out, accumulate, kernel, knobs):
    if din == "i8" and K % 64:
        K = 64 * ((K + 63) // 64)
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, gu.PATHS[kernel])
    run_and_check(M, K, N, din, out, 32, "padded", accumulate, seed=M + K + N)


# Whole 64 x 64 tiles and 128-byte K stages with 16-bit inputs: the
# small-tile ring kernel, forced, from one tile and one stage to long K
# (many refills of its 8-slot ring) and to more tiles than CUs.
RING = [(64, 64, 64), (64, 128, 192), (192, 448, 128), (320, 960, 128), (128, 4096, 64),
        (1024, 1024, 1024), (2048, 192, 2112)]


@pytest.mark.parametrize("pitch", ["contiguous", "padded"])
@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS[:3])
@pytest.mark.parametrize("M,K,N", RING)
def test_rect_ring_kernel(M, K, N, din, out, accumulate, pitch, knobs):
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_RING)
    s = 32 if din == "bf16" else 16
    run_and_check(M, K, N, din, out, s, pitch, accumulate, seed=M + 5 * K + 11 * N)


# Large ragged shapes (at least one 256 x 256 tile per CU): the full-tile
# kernel with the contracted index's partial last stage zero-padded in the
# kernel, and either its own edge tiles (N a whole number of 16-byte chunks)
# or the general kernel for the bottom rows and right columns.  All three
# dimensions ragged with edges in the kernel (4176: also for int8) or in
# strips (4173); edges in the kernel for 16-bit inputs and in strips for
# int8 (4104); only K; only M; a K tail of one element with one ragged
# column (int8: K below one stage, the general kernel alone).  Contiguous
# pitches that are not multiples of 16 bytes take the general kernel with
# 128 x 128 tiles, whole chunks loaded in 8-byte pieces (int8 K = 1000,
# bfloat16 N = 4100), 4-byte pieces (int8 K = 1004) or element by element
# (odd int8 or 16-bit pitches).
LARGE_RAGGED = [(4101, 1000, 4176), (4101, 1000, 4173), (4375, 1000, 4104), (4096, 1000, 4096),
                (4100, 1024, 4096), (4096, 33, 4097), (4101, 1004, 4100)]


@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("M,K,N", LARGE_RAGGED)
def test_rect_large_ragged_interior_and_edges(M, K, N, din, out, accumulate):
    s = 32 if din == "bf16" else 16
    run_and_check(M, K, N, din, out, s, "contiguous", accumulate, seed=M + K + N)


@pytest.mark.parametrize("N", [4176, 4173])
@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS)
def test_rect_large_ragged_padded_pitches(din, out, accumulate, N):
    s = 32 if din == "bf16" else 16
    run_and_check(4101, 1000, N, din, out, s, "padded", accumulate, seed=77 + N)


@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("accumulate", [False, True])
def test_rect_full_tiles_many_per_workgroup(din, out, accumulate, knobs):
    """The full-tile kernel's persistent loop with 3 workgroups for 12 tiles
    of 256 x 256 (each workgroup walks 4 tiles, reloading its ring)."""
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_FULL_TILE)
    knobs(tcu.TCU_KNOB_PP_GRID, 3)
    run_and_check(768, 512, 1024, din, out, 32, "padded", accumulate, seed=12)


@pytest.mark.parametrize("nsplit", [2, 3, 4, 7])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("accumulate", [False, True])
def test_rect_split_k(din, out, accumulate, nsplit, knobs):
    """Split-K on the full-tile kernel: the stages cut into nsplit ranges
    whose partial tiles are added into C atomically (after zeroing C when
    overwriting).  int32 stays bit-exact; a bfloat16 output is never split
    (rounded once), so it must pass the single-rounding check."""
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_FULL_TILE)
    knobs(tcu.TCU_KNOB_SPLIT_K, nsplit)
    run_and_check(512, 1344 if din != "i8" else 2688, 256, din, out, 32, "padded", accumulate,
                  seed=40 + nsplit)


@pytest.mark.parametrize("din,out", PAIRS)
def test_rect_split_k_many_items_per_workgroup(din, out, knobs):
    """Split-K items walked by a persistent grid of 5 workgroups: 6 tiles
    x 3 K ranges = 18 items, the first 16 in the permuted (XCD-grouped)
    order and the last 2 in their own."""
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_FULL_TILE)
    knobs(tcu.TCU_KNOB_PP_GRID, 5)
    knobs(tcu.TCU_KNOB_SPLIT_K, 3)
    run_and_check(512, 768 if din != "i8" else 1536, 768, din, out, 32, "padded", True,
                  seed=61)


# The tail split: tiles beyond the last whole round of the persistent grid
# cut into K ranges added atomically (binary32 and int32 outputs; C's tail
# tiles zeroed first when overwriting).  (M, N, grid, forced ranges):
# 10 tiles on 4 workgroups (2 tail tiles x 3 ranges, several rounds of split
# items), 12 tiles on 8 (4 x 4 = 16 split items in the XCD-grouped order).
@pytest.mark.parametrize("M,N,grid,ns", [(512, 1280, 4, 3), (768, 1024, 8, 4)])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("accumulate", [False, True])
def test_rect_tail_split(M, N, grid, ns, din, out, accumulate, knobs):
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_FULL_TILE)
    knobs(tcu.TCU_KNOB_PP_GRID, grid)
    knobs(tcu.TCU_KNOB_TAIL_SPLIT, ns)
    K = 31 * 64 // ES[din]                  # 31 stages: uneven ranges
    run_and_check(M, K, N, din, out, 32, "padded", accumulate, seed=M + N + ns)


@pytest.mark.parametrize("din,out", PAIRS)
def test_rect_tail_split_chosen_by_size(din, out, knobs):
    """Without forcing: 10 tiles on 4 workgroups and 64 stages give the 2
    tail tiles 2 ranges of 32 stages."""
    knobs(tcu.TCU_KNOB_GEMM_KERNEL, tcu.TCU_PATH_FULL_TILE)
    knobs(tcu.TCU_KNOB_PP_GRID, 4)
    run_and_check(512, 64 * 64 // ES[din], 1280, din, out, 32, "padded", False, seed=5)


@pytest.mark.parametrize("accumulate", [False, True])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("M,K,N", [(4101, 1000, 4176), (4375, 1000, 4104)])
def test_rect_large_ragged_tail_split(M, K, N, din, out, accumulate, knobs):
    """The ragged full-tile kernel with its tail tiles split 3 ways: edge
    tiles in the kernel (17 x 17 tiles) and, for int8 on the second shape,
    the 256-aligned interior (17 x 16 tiles) with the general kernel on the
    strips."""
    knobs(tcu.TCU_KNOB_TAIL_SPLIT, 3)
    s = 32 if din == "bf16" else 16
    run_and_check(M, K, N, din, out, s, "contiguous", accumulate, seed=M + K + N + 1)


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("M", [7, 16, 4099])
def test_rect_single_strip_is_the_native_call(M, s, din, out):
    """K = N = s with contiguous operands is one tall call (the native
    kernel), here accumulating; M below s is zero-padded."""
    tcu.tcu_reset_calls()
    run_and_check(M, s, s, din, out, s, "contiguous", True, seed=M + s)
    assert tcu.tcu_calls() == 1
    assert tcu.tcu_square_calls() == (M + s - 1) // s


@pytest.mark.parametrize("din,out", PAIRS)
def test_rect_k_zero(din, out):
    """K = 0: an empty sum.  Overwriting stores zeros; accumulating leaves C
    as it was (bit for bit)."""
    A = torch.empty(40, 0, dtype=inputs.TORCH_DTYPE[din])
    B = torch.empty(0, 24, dtype=inputs.TORCH_DTYPE[din])
    got = gu.run_rect(A, B, 16, din, out, 8, 24, 24)
    assert not np.any(np.asarray(got, dtype=np.float64))
    C0 = gu.c0_draw((40, 24), out, 3)
    got = gu.run_rect(A, B, 16, din, out, 8, 24, 24, C0=C0)
    assert np.array_equal(np.asarray(got), to_np_c0(C0, out))


def test_rect_empty_output_writes_nothing():
    A, B = gu.draw_pair((0, 64), (64, 32), "bf16", 1)
    got = gu.run_rect(A, B, 16, "bf16", "f32", 64, 32, 32)
    assert got.shape == (0, 32)
    A, B = gu.draw_pair((64, 64), (64, 0), "bf16", 2)
    got = gu.run_rect(A, B, 16, "bf16", "f32", 64, 8, 8)
    assert got.shape == (64, 0)


@pytest.mark.parametrize("s", [16, 32])
def test_rect_call_accounting(s):
    """ceil(K/s) * ceil(N/s) calls of ceil(M/s) square calls each."""
    M, K, N = 100, 130, 70
    tcu.tcu_reset_calls()
    run_and_check(M, K, N, "bf16", "f32", s, "padded", False, seed=9)
    calls = -(-K // s) * -(-N // s)
    assert tcu.tcu_calls() == calls
    assert tcu.tcu_square_calls() == calls * -(-M // s)
    assert tcu.tcu_work() == calls * -(-M // s) * s * s


def test_rect_int32_wraps_around():
    """The accumulating int32 sum wraps modulo 2^32 (documented)."""
    M, K, N = 64, 64, 64
    A = torch.full((M, K), 100, dtype=torch.int8)
    B = torch.full((K, N), 100, dtype=torch.int8)        # A*B = 640000 per entry
    C0 = torch.full((M, N), 2 ** 31 - 1000, dtype=torch.int32)
    got = gu.run_rect(A, B, 16, "i8", "i32", K, N, N, C0=C0)
    want = compare.wrap_i32(np.full((M, N), 2 ** 31 - 1000 + 640000, dtype=np.int64))
    assert np.array_equal(got.astype(np.int64), want)
    assert int(got[0, 0]) < 0


@pytest.mark.parametrize("din,out", PAIRS)
def test_rect_split_k_accumulation_composes(din, out):
    """C = A[:, :K1] B[:K1] then C += A[:, K1:] B[K1:] (Theorem 2's sum over
    strips, done in two calls on views of the same arrays).  Each call is
    checked against the oracle on its own (the second with the first's
    stored result as C0); the end result is bit-exact with the one-call
    product for int8 and within tolerance of it for binary32 outputs.  (A
    bfloat16 output is rounded after each call, so there the composition is
    only checked call by call.)"""
    M, K, N, K1 = 300, 200, 140, 96
    A, B = gu.draw_pair((M, K), (K, N), din, 77)
    dA = gu.pitched_input(A, aligned_pitch(K, ES[din]), din)
    dB = gu.pitched_input(B, aligned_pitch(N, ES[din]), din)
    C = torch.empty(M, N, dtype=gu.out_dtype(out), device=gu.DEV)
    tcu.tcu_set_unit(16)
    lda, ldb = dA.stride(0), dB.stride(0)
    tcu.tcu_gemm_rect(dA[:, :K1], lda, dB[:K1], ldb, C, N, M, K1, N)
    torch.cuda.synchronize()
    first = gu.to_np(C).copy()
    tcu.tcu_gemm_rect(dA[:, K1:], lda, dB[K1:], ldb, C, N, M, K - K1, N, tcu.TCU_ACCUMULATE)
    torch.cuda.synchronize()
    got = gu.to_np(C)
    Ab, Bb = inputs.bits(A), inputs.bits(B)
    compare.check(din, out, Ab[:, :K1], Bb[:K1], first)
    compare.check(din, out, np.ascontiguousarray(Ab[:, K1:]), np.ascontiguousarray(Bb[K1:]),
                  got, C0=first)
    if din == "i8":
        full = gu.run_rect(A, B, 16, din, out, K, N, N)
        assert np.array_equal(got, full)
    if out != "bf16":
        compare.check(din, out, Ab, Bb, got)


@pytest.mark.parametrize("s", [16, 32])
def test_rect_d_function_in_place_blocks(s):
    """The D function X <- X + Y*Z on disjoint blocks of one bfloat16 array
    (blocks as in the recursive Gaussian elimination and transitive-closure
    algorithms), through strided views of that array."""
    n, b = 256, 64
    g = torch.Generator().manual_seed(31)
    host = inputs.draw((n, n), "bf16", "normal", g)
    X0 = host.clone()
    dev = host.to(gu.DEV)
    blocks = [((0, 64), (0, 0), (64, 64)),      # X = (0,1), Y = (0,0), Z = (1,1)
              ((128, 0), (128, 64), (64, 0)),   # X = (2,0), Y = (2,1), Z = (1,0)
              ((192, 192), (192, 128), (128, 192))]
    for (xr, xc), (yr, yc), (zr, zc) in blocks:
        X = dev[xr:xr + b, xc:xc + b]
        Y = dev[yr:yr + b, yc:yc + b]
        Z = dev[zr:zr + b, zc:zc + b]
        tcu.tcu_set_unit(s)
        tcu.tcu_gemm_rect(Y, n, Z, n, X, n, b, b, b, tcu.TCU_ACCUMULATE)
    torch.cuda.synchronize()
    got = dev.cpu()
    bits = lambda t: inputs.bits(t.contiguous())
    for (xr, xc), (yr, yc), (zr, zc) in blocks:
        blk = lambda t, r, c: t[r:r + b, c:c + b]
        compare.check("bf16", "bf16", bits(blk(X0, yr, yc)), bits(blk(X0, zr, zc)),
                      bits(blk(got, xr, xc)), C0=bits(blk(X0, xr, xc)))
    # every element outside the three X blocks is untouched
    mask = torch.ones(n, n, dtype=torch.bool)
    for (xr, xc), _, _ in blocks:
        mask[xr:xr + b, xc:xc + b] = False
    assert torch.equal(got.view(torch.int16)[mask], X0.view(torch.int16)[mask])


# Corollary 1 at full size, every element: sqrt(n) x r times r x sqrt(n)
# with r below and above sqrt(n), plus the benchmark's rectangular workloads
# exactly as the benchmark runs them (contiguous operands).
COR1 = [
    # (M = N = sqrt(n), K = r, in, out, accumulate)
    (8192, 1024, "i8", "i32", False),
    (2048, 32768, "bf16", "bf16", True),
    (4096, 4096 + 32, "f16", "f32", True),
]


@pytest.mark.parametrize("M,K,din,out,accumulate", COR1)
def test_rect_corollary1_full(M, K, din, out, accumulate):
    N = M
    A, B = gu.draw_pair((M, K), (K, N), din, 5)
    C0 = gu.c0_draw((M, N), out, 6) if accumulate else None
    got = gu.run_rect(A, B, 32, din, out, K, N, N, C0=C0)
    compare.check(din, out, inputs.bits(A), inputs.bits(B), got,
                  C0=None if C0 is None else to_np_c0(C0, out))


@pytest.mark.parametrize("name", sorted(inputs.RECT_WORKLOADS))
def test_rect_workload_full(name):
    sp = inputs.RECT_WORKLOADS[name]
    M, K, N = sp["M"], sp["K"], sp["N"]
    A, B = inputs.make_inputs(sp)
    C0 = inputs.make_c0(sp) if sp["acc"] else None
    got = gu.run_rect(A, B, sp["s"], sp["dtype"], sp["out"], K, N, N, C0=C0)
    rep = compare.check(sp["dtype"], sp["out"], inputs.bits(A), inputs.bits(B), got,
                        C0=None if C0 is None else to_np_c0(C0, sp["out"]))
    print(name, rep)
