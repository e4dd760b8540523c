"""Parity checks of GPU results against the oracle -- TEST INFRASTRUCTURE ONLY.

Tolerances (the paper fixes no precision; these are the stated bar):
  * floating point: relative Frobenius error <= 1e-3 AND, elementwise,
    |err_ij| <= 1e-2 * (|A| |B|)_ij, against the binary64 oracle;
  * bfloat16 output: relative Frobenius error <= 1e-3 against the oracle
    rounded once (nearest-even) to bfloat16 -- against the unrounded oracle
    the output format alone costs about 1.7e-3 on N(0,1) data -- and the
    elementwise bound above against the unrounded binary64 oracle (bfloat16
    rounding alone is at most 2^-9 |c|).  In addition every element g must
    be a nearest rounding of some value within the binary32 summation bound
    of the exact sum s:  |g - s| <= ulp(g)/2 + K 2^-23 (|A| |B|)_ij, which
    catches a wrong rounding step (truncation, double rounding across
    binades) while allowing the legitimate one-step differences that
    cancellation in a K-term binary32 sum produces;
  * int8 -> int32: bit-exact.
(|A| |B|) is the oracle's product of the operands with their sign bits
cleared.
"""
from __future__ import annotations

import numpy as np

from . import decode_out, f64_to_bf16, bf16_to_f64, mm, mm_acc, poly_eval

REL_FROB = 1e-3
ELEM = 1e-2


def abs_bits(x: np.ndarray) -> np.ndarray:
    """|x| of 16-bit float bit patterns (sign bit cleared)."""
    return np.ascontiguousarray(x).view(np.uint16) & np.uint16(0x7FFF)


def float_report(got: np.ndarray, ref: np.ndarray, absab: np.ndarray) -> dict:
    got = np.asarray(got, dtype=np.float64)
    err = np.abs(got - ref)
    denom = np.linalg.norm(ref)
    rel = float(np.linalg.norm(got - ref) / denom) if denom > 0 else float(np.linalg.norm(got - ref))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(absab > 0, err / absab, np.where(err > 0, np.inf, 0.0))
    return {"rel_frob": rel, "max_elem_ratio": float(ratio.max(initial=0.0)),
            "max_abs_err": float(err.max(initial=0.0))}


def check_float(got, ref, absab) -> dict:
    rep = float_report(got, ref, absab)
    assert rep["rel_frob"] <= REL_FROB, rep
    assert rep["max_elem_ratio"] <= ELEM, rep
    return rep


def bf16_ulp_distance(a_bits: np.ndarray, b_bits: np.ndarray) -> np.ndarray:
    """Distance in bfloat16 steps between two arrays of finite bf16 patterns."""
    def ordered(x):
        x = np.asarray(x, dtype=np.uint16).astype(np.int64)
        mag = x & 0x7FFF
        return np.where(x & 0x8000, -mag, mag)
    return np.abs(ordered(a_bits) - ordered(b_bits))


def bf16_spacing(x: np.ndarray) -> np.ndarray:
    """Gap between consecutive bfloat16 values in the binade of |x|."""
    ax = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    e = np.maximum(e, -126.0)
    return np.where(ax > 0, np.ldexp(1.0, (e - 7).astype(np.int64)), 2.0 ** -133)


def check_bf16(got_bits, ref64, absab, K: int) -> dict:
    got_bits = np.asarray(got_bits).view(np.uint16)
    ref_bits = f64_to_bf16(ref64)
    ulps = bf16_ulp_distance(got_bits, ref_bits)
    got = bf16_to_f64(got_bits)
    rounded = bf16_to_f64(ref_bits)
    rep_r = float_report(got, rounded, absab)
    rep_u = float_report(got, ref64, absab)
    slack = np.abs(got - ref64) - (0.5 * bf16_spacing(got) + K * 2.0 ** -23 * absab)
    rep = {"max_ulps_vs_rounded": int(ulps.max(initial=0)),
           "frac_off_by_one": float((ulps > 0).mean()) if ulps.size else 0.0,
           "rel_frob_vs_rounded": rep_r["rel_frob"],
           "rel_frob_vs_unrounded": rep_u["rel_frob"],
           "max_elem_ratio_vs_unrounded": rep_u["max_elem_ratio"],
           "rounding_violations": int((slack > 0).sum())}
    assert np.all(np.isfinite(got)), rep
    assert rep["rounding_violations"] == 0, rep
    assert rep["rel_frob_vs_rounded"] <= REL_FROB, rep
    assert rep["max_elem_ratio_vs_unrounded"] <= ELEM, rep
    return rep


def check_exact(got, ref) -> dict:
    got = np.asarray(got, dtype=np.int64)
    mism = int((got != ref).sum())
    assert mism == 0, f"{mism} int mismatches"
    return {"mismatches": 0}


def wrap_i32(x: np.ndarray) -> np.ndarray:
    """Exact integers reduced to int32 two's complement (wrap-around)."""
    x = np.asarray(x, dtype=np.int64)
    return ((x + 2 ** 31) % 2 ** 32) - 2 ** 31


def check(dtype_in: str, dtype_out: str, A_bits, B_bits, got, rows=None, C0=None) -> dict:
    """Compare a GPU result (numpy; bf16 output as uint16 bits) with the oracle
    on the given rows of A (all rows when None).

    C0: the stored output before an accumulating call (full matrix, stored
    values: float32, bf16 bits or int32); the reference is then C0 + A*B,
    the binary32 (or int32) addition of C0 counting as one more term of
    the sum in the error bounds, whose magnitude term becomes
    |A| |B| + |C0|.  int32 results are compared modulo 2^32, the documented
    wrap-around of the accumulating form."""
    if C0 is None:
        ref = mm(A_bits, B_bits, dtype_in, rows=rows)
    else:
        ref = mm_acc(A_bits, B_bits, C0, dtype_in, dtype_out, rows=rows)
    if dtype_in == "i8":
        return check_exact(got, wrap_i32(ref) if C0 is not None else ref)
    absab = mm(abs_bits(A_bits), abs_bits(B_bits), dtype_in, rows=rows)
    K = np.asarray(A_bits).shape[1]
    if C0 is not None:
        c0 = np.abs(decode_out(C0, dtype_out))
        absab = absab + (c0 if rows is None else c0[np.asarray(rows, dtype=np.int64)])
        K += 1
    if dtype_out == "bf16":
        return check_bf16(got, ref, absab, K=K)
    return check_float(got, ref, absab)


def poly_bound(dtype_in: str, n: int, s: int) -> float:
    """Relative-to-magnitude error bound of the batch polynomial evaluation
    (Theorem 11) as the unit computes it, times a safety factor of 4:
      * X = X_hi + X_lo as two bfloat16 words (for both input types; the
        binary16 coefficients are split exactly into two bfloat16 words)
        leaves a residual of at most 2^-17 |x^k|: hi is x^k rounded to
        nearest with 8 significant bits, so the remainder is at most 2^-8 of
        the power of two 2^e at or below |x^k|, and strictly below it unless
        it is exactly that power of two (then lo holds it exactly); a
        remainder below 2^(e-8) rounds to 8 significant bits with an error of
        at most 2^(e-17);
      * every power is a chain of at most 2 log2(s) + s binary32 products,
        the block weights y^(s J) a chain of n/s^2 more;
      * the unit's sums run over s products, the combine over s + n/s^2
        terms plus two cross-lane additions;
    each binary32 operation adding at most 2^-24 of the magnitude sum
    sum_h |a_h| |x|^h."""
    if dtype_in not in ("f16", "bf16"):
        raise ValueError("polynomial evaluation takes f16 or bf16 inputs")
    split = 2.0 ** -17
    ops = 2 * 6 + s + s + 2 * (n // (s * s) + 1) + 8
    return 4.0 * (split + ops * 2.0 ** -24)


def check_poly(dtype_in: str, dtype_out: str, coef_bits, pt_bits, got, s: int,
               idx=None) -> dict:
    """Compare GPU polynomial values (numpy float32, or bf16 bits for a
    bfloat16 output) with the oracle: elementwise
    |g - A(x)| <= poly_bound * sum_h |a_h||x|^h (+ half a bfloat16 ulp of
    g for a bfloat16 output), and relative Frobenius error <= 1e-3 against
    the exact values (1e-3 + 2^-9 for a bfloat16 output: the format's own
    rounding; a bfloat16 value is also checked elementwise, above, to be a
    nearest rounding of a value within the bound).
    idx: the point indices `got` holds (all points when None)."""
    pts = np.ascontiguousarray(pt_bits).view(np.uint16)
    if idx is not None:
        pts = pts[np.asarray(idx, dtype=np.int64)]
    val, mag = poly_eval(coef_bits, pts, dtype_in)
    n = np.asarray(coef_bits).size
    if dtype_out == "bf16":
        g = bf16_to_f64(np.asarray(got).view(np.uint16))
        extra = 0.5 * bf16_spacing(g)
    else:
        g = np.asarray(got, dtype=np.float64)
        extra = 0.0
    err = np.abs(g - val)
    allow = poly_bound(dtype_in, n, s) * mag + extra
    denom = np.linalg.norm(val)
    rel = float(np.linalg.norm(g - val) / denom) if denom > 0 else float(np.linalg.norm(g - val))
    # one nearest rounding to bfloat16 moves every value by at most 2^-9 of
    # itself, so the output format adds at most 2^-9 to the relative
    # Frobenius error against the exact values
    rel_bar = REL_FROB + (2.0 ** -9 if dtype_out == "bf16" else 0.0)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(mag > 0, err / mag, np.where(err > 0, np.inf, 0.0))
    rep = {"rel_frob": rel, "max_err_over_magnitude": float(ratio.max(initial=0.0)),
           "bound": poly_bound(dtype_in, n, s), "violations": int((err > allow).sum())}
    assert np.all(np.isfinite(g)), rep
    assert rep["violations"] == 0, rep
    assert rel <= rel_bar, rep
    return rep


def dft_sample_freqs(n: int, seed: int = 0, k: int = 64) -> np.ndarray:
    """Output frequencies a large transform is checked on against the
    definition: 0, 1, 2, n/2 - 1, n/2, n/2 + 1, n - 2, n - 1 and k seeded
    random ones (sorted, distinct, all of them when n is small)."""
    if n <= k + 8:
        return np.arange(n, dtype=np.int64)
    fixed = np.array([0, 1, 2, n // 2 - 1, n // 2, n // 2 + 1, n - 2, n - 1], dtype=np.int64)
    rng = np.random.default_rng(seed)
    ks = set(fixed.tolist())
    while len(ks) < k + fixed.size:
        ks.add(int(rng.integers(0, n)))
    return np.array(sorted(ks), dtype=np.int64)


# Largest n whose whole transform the definition computes (O(n^2) per vector).
DFT_FULL_MAX = 1024


def _dft_report(got: np.ndarray, ref: np.ndarray, mag: np.ndarray) -> dict:
    err = np.abs(got - ref)
    den = np.linalg.norm(ref, axis=1)
    rel = np.where(den > 0, np.linalg.norm(got - ref, axis=1) / np.where(den > 0, den, 1), 0.0)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(mag > 0, err / mag, np.where(err > 0, np.inf, 0.0))
    return {"max_rel_frob": float(rel.max(initial=0.0)),
            "max_err_over_l1": float(ratio.max(initial=0.0))}


def check_dft(x: np.ndarray, got: np.ndarray, ref: np.ndarray | None = None,
              ks: np.ndarray | None = None, fft_extra: bool = True) -> dict:
    """Compare a GPU DFT (complex, rows = vectors) with the binary64 oracle:
    relative Frobenius error <= 1e-3 per vector, and elementwise
    |err_k| <= 1e-2 * sum_j |x_j| (the magnitude bound: |W| = 1).

    The reference is the definition y[k] = sum_j x[j] w^(jk): on every
    output for n <= 1024, else on the frequencies ks (dft_sample_freqs(n)
    when None; the relative Frobenius error is then taken over those
    outputs).  For n > 1024 the whole transform is also compared with
    numpy's binary64 FFT when fft_extra is set, an extra check only.
    ref: the definition at ks (or everywhere) when already computed."""
    from . import dft, dft_direct, dft_direct_at
    x = np.asarray(x, dtype=np.complex128).reshape(-1, np.asarray(x).shape[-1])
    got = np.asarray(got, dtype=np.complex128).reshape(x.shape)
    n = x.shape[1]
    assert np.all(np.isfinite(got)), "non-finite DFT output"
    mag = np.sum(np.abs(x), axis=1, keepdims=True)
    if ks is None and n > DFT_FULL_MAX:
        ks = dft_sample_freqs(n)
    if ks is None:
        if ref is None:
            ref = dft_direct(x)
        rep = _dft_report(got, np.asarray(ref).reshape(x.shape), mag)
        rep["freqs_checked"] = n
    else:
        ks = np.asarray(ks, dtype=np.int64)
        if ref is None:
            ref = dft_direct_at(x, ks)
        rep = _dft_report(got[:, ks], np.asarray(ref).reshape(x.shape[0], ks.size), mag)
        rep["freqs_checked"] = int(ks.size)
    assert rep["max_rel_frob"] <= REL_FROB, rep
    assert rep["max_err_over_l1"] <= ELEM, rep
    if fft_extra and n > DFT_FULL_MAX:
        extra = _dft_report(got, dft(x), mag)
        rep["fft_max_rel_frob"] = extra["max_rel_frob"]
        assert extra["max_rel_frob"] <= REL_FROB, rep
        assert extra["max_err_over_l1"] <= ELEM, rep
    return rep
