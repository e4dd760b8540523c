"""Pins of the oracle's batch polynomial evaluation (Theorem 11, Section 4.8)
against what the mathematics fixes (CPU only).

The oracle evaluates A(x) = sum_h a_h x^h term by term in binary64 on the
decoded 16-bit inputs.  It is checked by routes that do not reuse its code:
exact rational brute force on small cases, closed forms (geometric series,
binomial expansion, a Chebyshev polynomial against cos(n arccos x)), the
special points 0, 1 and -1, and a group of plausible mistakes (reversed
coefficients, powers shifted by one, a dropped last term) that the pins must
reject.
"""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

from paper_1908_06649_amd import inputs

U64 = 2.0 ** -53


def to_bits(vals, dtype):
    t = torch.tensor(vals, dtype=torch.float32).to(inputs.TORCH_DTYPE[dtype])
    return inputs.bits(t)


def exact(bits16: int, dtype: str) -> Fraction:
    if dtype == "f16":
        return Fraction(struct.unpack("<e", struct.pack("<H", bits16))[0])
    return Fraction(struct.unpack("<f", struct.pack("<I", bits16 << 16))[0])


def brute(coef_bits, pt_bits, dtype):
    a = [exact(int(b), dtype) for b in coef_bits]
    out = []
    for pb in pt_bits:
        x = exact(int(pb), dtype)
        out.append(sum(ah * x ** h for h, ah in enumerate(a)))
    return out


def within(got, want: Fraction, mag: float, n: int) -> bool:
    """|got - want| <= 2 n u64 mag (+ a tiny absolute term for mag = 0)."""
    return abs(Fraction(float(got)) - want) <= Fraction(2 * n * U64 * mag) + Fraction(1, 2 ** 1000)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("n", [1, 2, 5, 16, 33])
def test_poly_vs_exact_rational(oracle_mod, dtype, n):
    g = torch.Generator().manual_seed(n * 3 + (dtype == "bf16"))
    coef = inputs.bits(inputs.draw((n,), dtype, "normal", g))
    pts = inputs.bits(inputs.draw((9,), dtype, "uniform", g))
    val, mag = oracle_mod.poly_eval(coef, pts, dtype)
    for v, m, w in zip(val, mag, brute(coef, pts, dtype)):
        assert within(v, w, m, n)


def test_poly_geometric_series(oracle_mod):
    """a_h = 1: A(x) = (1 - x^n) / (1 - x)."""
    n = 50
    coef = to_bits([1.0] * n, "bf16")
    xs = [-0.875, -0.5, -0.0625, 0.25, 0.5, 0.9375]
    pts = to_bits(xs, "bf16")
    val, mag = oracle_mod.poly_eval(coef, pts, "bf16")
    for v, m, pb in zip(val, mag, pts):
        x = exact(int(pb), "bf16")
        assert within(v, (1 - x ** n) / (1 - x), m, n)


def test_poly_binomial(oracle_mod):
    """a_h = C(9, h): A(x) = (1 + x)^9 (every coefficient <= 126 is exact in
    both 16-bit formats)."""
    for dtype in ("f16", "bf16"):
        coef = to_bits([math.comb(9, h) for h in range(10)], dtype)
        xs = [-1.5, -1.0, -0.3, 0.0, 0.7, 1.25, 2.0]
        pts = to_bits(xs, dtype)
        val, mag = oracle_mod.poly_eval(coef, pts, dtype)
        for v, m, pb in zip(val, mag, pts):
            x = exact(int(pb), dtype)
            assert within(v, (1 + x) ** 9, m, 10)


def test_poly_chebyshev_t8(oracle_mod):
    """T_8(x) = 128x^8 - 256x^6 + 160x^4 - 32x^2 + 1 = cos(8 arccos x) on [-1, 1]."""
    coef = to_bits([1, 0, -32, 0, 160, 0, -256, 0, 128], "bf16")
    xs = np.linspace(-1.0, 1.0, 41)
    pts = to_bits(xs.tolist(), "bf16")
    val, mag = oracle_mod.poly_eval(coef, pts, "bf16")
    x = oracle_mod.bf16_to_f64(pts)
    ref = np.cos(8 * np.arccos(x))
    assert np.all(np.abs(val - ref) <= 1e-12 * mag)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_poly_special_points(oracle_mod, dtype):
    g = torch.Generator().manual_seed(11)
    n = 40
    coef = inputs.bits(inputs.draw((n,), dtype, "normal", g))
    a = oracle_mod.decode(coef, dtype)
    pts = to_bits([0.0, 1.0, -1.0], dtype)
    val, mag = oracle_mod.poly_eval(coef, pts, dtype)
    assert val[0] == a[0] and mag[0] == abs(a[0])           # x = 0 (0^0 = 1)
    assert abs(val[1] - math.fsum(a)) <= 2 * n * U64 * mag[1]
    alt = math.fsum(a[h] * (-1) ** h for h in range(n))
    assert abs(val[2] - alt) <= 2 * n * U64 * mag[2]
    assert mag[1] == pytest.approx(math.fsum(np.abs(a)), rel=1e-15)


def test_poly_magnitude_is_abs_polynomial(oracle_mod):
    """sum_h |a_h| |x|^h is the value of the polynomial with |a_h| at |x|."""
    g = torch.Generator().manual_seed(12)
    coef = inputs.bits(inputs.draw((70,), "bf16", "normal", g))
    pts = inputs.bits(inputs.draw((50,), "bf16", "uniform", g))
    val, mag = oracle_mod.poly_eval(coef, pts, "bf16")
    absval, _ = oracle_mod.poly_eval(coef & np.uint16(0x7FFF), pts & np.uint16(0x7FFF), "bf16")
    assert np.allclose(mag, absval, rtol=1e-14, atol=0)
    assert np.all(np.abs(val) <= mag * (1 + 1e-14))


def test_poly_empty_and_rejects(oracle_mod):
    val, mag = oracle_mod.poly_eval(np.zeros(0, np.uint16), to_bits([0.5, 2.0], "bf16"), "bf16")
    assert np.all(val == 0) and np.all(mag == 0)
    with pytest.raises(ValueError):
        oracle_mod.poly_eval(np.zeros(3, np.int8), np.zeros(3, np.int8), "i8")


@pytest.mark.parametrize("mistake", ["reversed", "shifted_power", "dropped_last"])
def test_poly_pins_catch_planted_mistakes(oracle_mod, mistake):
    """An oracle with a plausible indexing mistake -- emulated by feeding it
    transformed coefficients -- fails the exact brute-force pin."""
    dtype, n = "bf16", 12
    g = torch.Generator().manual_seed(99)
    coef = inputs.bits(inputs.draw((n,), dtype, "normal", g))
    pts = to_bits([0.5, -0.75, 0.875], dtype)
    if mistake == "reversed":
        bad = coef[::-1].copy()
    elif mistake == "shifted_power":                   # uses x^(h+1) for a_h
        bad = np.concatenate([np.zeros(1, np.uint16), coef])
    else:
        bad = coef[:-1].copy()
    val, mag = oracle_mod.poly_eval(bad, pts, dtype)
    want = brute(coef, pts, dtype)
    assert not all(within(v, w, m, n) for v, m, w in zip(val, mag, want))
