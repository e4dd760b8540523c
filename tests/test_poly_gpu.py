"""GPU parity of batch polynomial evaluation (tcu_poly_eval, Theorem 11,
Section 4.8) against the CPU oracle's binary64 evaluation of the definition,
through the C ABI.

The bar (oracle/compare.py check_poly): every value within a derived bound
times sum_h |a_h||x|^h, and relative Frobenius error <= 1e-3.  Small-integer
cases, where every power and sum is exact in binary32, must match bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import bf16_to_f64, compare, poly_eval
from paper_1908_06649_amd import inputs, tcu

import gpu_util as gu

pytestmark = pytest.mark.gpu

PAIRS = [("f16", "f32"), ("bf16", "f32"), ("bf16", "bf16")]


def run_poly(coef: torch.Tensor, pts: torch.Tensor, s: int, out: str, guard=True):
    n, p = coef.numel(), pts.numel()
    buf, o = gu.sentinel_buffer(p, gu.out_dtype(out))
    tcu.tcu_set_unit(s)
    tcu.tcu_poly_eval(coef.to(gu.DEV), n, pts.to(gu.DEV), p, o)
    torch.cuda.synchronize()
    if guard:
        assert gu.guard_intact(buf, p), "wrote past the end of out"
    return gu.to_np(o)


def draw(n, p, din, seed, coef_dist="normal"):
    g = torch.Generator().manual_seed(seed)
    return inputs.draw((n,), din, coef_dist, g), inputs.draw((p,), din, "uniform", g)


SHAPES = [(1, 1), (5, 17), (16, 16), (64, 100), (256, 1000), (1000, 1000), (1024, 4096),
          (4099, 333), (5000, 2049), (20000, 64)]


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("din,out", PAIRS)
@pytest.mark.parametrize("n,p", SHAPES)
def test_poly_shapes(n, p, din, out, s):
    coef, pts = draw(n, p, din, seed=n * 13 + p + s)
    got = run_poly(coef, pts, s, out)
    compare.check_poly(din, out, inputs.bits(coef), inputs.bits(pts), got, s)


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("din", ["f16", "bf16"])
def test_poly_small_integers_exact(din, s):
    """Points and coefficients in {-2..2} with n <= 12 (one block column), and
    points in {-1, 0, 1} with n spanning several blocks: every power, product
    and sum is exact in binary32, so the values equal the oracle's exactly."""
    g = torch.Generator().manual_seed(5)
    coef = torch.randint(-2, 3, (12,), generator=g).to(inputs.TORCH_DTYPE[din])
    pts = torch.randint(-2, 3, (300,), generator=g).to(inputs.TORCH_DTYPE[din])
    pts[:5] = torch.tensor([-2, -1, 0, 1, 2]).to(pts.dtype)
    got = run_poly(coef, pts, s, "f32")
    want, _ = poly_eval(inputs.bits(coef), inputs.bits(pts), din)
    assert np.array_equal(got.astype(np.float64), want)
    coef = torch.randint(-2, 3, (3 * s * s + 7,), generator=g).to(inputs.TORCH_DTYPE[din])
    pts = torch.randint(-1, 2, (1000,), generator=g).to(inputs.TORCH_DTYPE[din])
    got = run_poly(coef, pts, s, "f32")
    want, _ = poly_eval(inputs.bits(coef), inputs.bits(pts), din)
    assert np.array_equal(got.astype(np.float64), want)


def test_poly_closed_forms():
    """Geometric series and (1 + x)^9 through the GPU path, against the
    closed forms evaluated in binary64."""
    n = 3000
    pts = torch.linspace(-0.99, 0.99, 777).to(torch.bfloat16)
    x = pts.to(torch.float64).numpy()
    got = run_poly(torch.ones(n, dtype=torch.bfloat16), pts, 32, "f32")
    ref = (1 - x ** n) / (1 - x)
    assert np.all(np.abs(got - ref) <= 1e-5 * np.abs(1 / (1 - np.abs(x))) + 1e-6)
    binom = torch.tensor([1, 9, 36, 84, 126, 126, 84, 36, 9, 1], dtype=torch.bfloat16)
    got = run_poly(binom, pts, 16, "f32")
    assert np.all(np.abs(got - (1 + x) ** 9) <= 1e-5 * (1 + np.abs(x)) ** 9)


@pytest.mark.parametrize("s", [16, 32])
def test_poly_short_polynomial_large_points(s):
    """n < s with |x| = 2..8 (bfloat16): the powers a degree-5 polynomial
    needs stay small, and the unused powers of the unit's padding must not
    overflow into the result."""
    coef = torch.tensor([1, -2, 0.5, 3, -1, 0.25], dtype=torch.bfloat16)
    pts = torch.tensor([2, -3, 4, -5, 8, 0.5, -1], dtype=torch.bfloat16)
    got = run_poly(coef, pts, s, "f32")
    compare.check_poly("bf16", "f32", inputs.bits(coef), inputs.bits(pts), got, s)


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("din,out", PAIRS)
def test_poly_sparse_high_powers_small_points(din, out, s):
    """Only the highest power of a block nonzero (a_(s-1) = 1, and a_h for
    h = -1 mod s in a longer polynomial), points with 0.1 <= |x| < 1: the
    value is carried by x^(s-1) alone, far below binary16's normal range
    (2^-14) for most points, yet every value must meet the bound relative to
    sum_h |a_h||x|^h.  binary16 X words would lose these terms entirely."""
    g = torch.Generator().manual_seed(41 + s)
    mag = 0.1 + 0.9 * torch.rand(3000, generator=g)
    sign = torch.where(torch.rand(3000, generator=g) < 0.5, -1.0, 1.0)
    pts = (mag * sign).to(inputs.TORCH_DTYPE[din])
    for n in (s, 3 * s * s):
        coef = torch.zeros(n)
        coef[s - 1::s] = 1.0
        coef = coef.to(inputs.TORCH_DTYPE[din])
        got = run_poly(coef, pts, s, out)
        rep = compare.check_poly(din, out, inputs.bits(coef), inputs.bits(pts), got, s)
        print(din, out, s, n, rep)
    # the advisor's example: a_31 = 1 at x = 0.5 is exactly 2^-31
    coef = torch.zeros(s)
    coef[s - 1] = 1.0
    got = run_poly(coef.to(inputs.TORCH_DTYPE[din]),
                   torch.tensor([0.5, -0.5, 0.25]).to(inputs.TORCH_DTYPE[din]), s, out)
    want = np.array([0.5, -0.5, 0.25]) ** (s - 1)
    val = bf16_to_f64(got) if out == "bf16" else np.asarray(got, dtype=np.float64)
    assert np.all(np.abs(val - want) <= 2.0 ** -8 * np.abs(want)), (val, want)


@pytest.mark.parametrize("din,out", PAIRS)
def test_poly_no_coefficients_gives_zeros(din, out):
    pts = torch.linspace(-1, 1, 50).to(inputs.TORCH_DTYPE[din])
    got = run_poly(torch.empty(0, dtype=inputs.TORCH_DTYPE[din]), pts, 32, out)
    assert not np.any(np.asarray(got, dtype=np.float64))


def test_poly_no_points_is_a_noop():
    tcu.tcu_reset_calls()
    coef = torch.ones(64, dtype=torch.bfloat16, device=gu.DEV)
    tcu.tcu_set_unit(32)
    tcu.tcu_poly_eval(coef, 64, torch.empty(0, dtype=torch.bfloat16, device=gu.DEV), 0,
                      torch.empty(0, dtype=torch.float32, device=gu.DEV))
    assert tcu.tcu_calls() == 0


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("din,per_block", [("bf16", 2), ("f16", 4)])
def test_poly_call_accounting(s, din, per_block):
    """Each of the n/m calls is issued for X_hi and X_lo, and for binary16
    coefficients also for c_hi and c_lo."""
    n, p = 5000, 700
    coef, pts = draw(n, p, din, 3)
    tcu.tcu_reset_calls()
    run_poly(coef, pts, s, "f32")
    calls = per_block * -(-n // (s * s))
    assert tcu.tcu_calls() == calls
    assert tcu.tcu_square_calls() == calls * -(-p // s)


def test_poly_deterministic():
    coef, pts = draw(4096, 5000, "bf16", 8)
    a = run_poly(coef, pts, 32, "f32")
    b = run_poly(coef, pts, 32, "f32")
    assert np.array_equal(a, b)


@pytest.mark.parametrize("name", sorted(inputs.POLY_WORKLOADS))
def test_poly_workload_all_points(name):
    sp = inputs.POLY_WORKLOADS[name]
    coef, pts = inputs.make_poly_inputs(sp)
    got = run_poly(coef, pts, sp["s"], sp["out"])
    rep = compare.check_poly(sp["dtype"], sp["out"], inputs.bits(coef), inputs.bits(pts),
                             got, sp["s"])
    print(name, rep)
