"""CPU oracle for the (m,l)-TCU hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package; the GPU library and its Python binding never import it.  It wraps
``liboracle.so`` (built from ``tcu_oracle.c`` by ``oracle/build.py``) with
numpy in/out:

* ``mm(A, B, dtype, rows=None)`` -- the plain product ``C = A*B`` that both
  the native tensor-unit call (Section 3, model definition) and the blocked
  multiplication of Theorem 2 (Section 4.1) compute.  ``A`` and ``B`` hold the
  stored bit patterns (uint16 for 'f16'/'bf16', int8 for 'i8'); the result is
  float64 (floating point) or int64 (exact integer).  ``rows`` selects rows of
  A so that large cases can be checked on sampled rows.
* ``f16_to_f64``, ``bf16_to_f64`` -- format decoders.
* ``f64_to_bf16`` -- one-step round-to-nearest-even to bfloat16 bit patterns.
* ``poly_eval(coef, points, dtype)`` -- A(x) = sum_h a_h x^h at every point
  (Theorem 11, Section 4.8), in binary64 on the decoded 16-bit inputs, with
  the magnitude sum sum_h |a_h| |x|^h.
* ``transitive_closure(d)`` -- reachability by paths of >= 1 edge from an
  n x n 0/1 adjacency matrix (Section 4.3), by the in-place iterative
  algorithm the section starts from (k outermost, then i, then j).
* ``dft_direct(x)`` -- the DFT by its definition y = x^T W, W[r][c] =
  exp(-2 pi i r c / n) (Section 4.5), O(n^2) per vector, binary64;
  ``dft_direct_at(x, ks)`` -- the same definition at chosen output
  frequencies only (O(n) each), which checks vectors of any length on a
  sample of their outputs; ``dft(x)`` -- the whole transform through numpy's
  binary64 FFT, an extra check at large sizes only (pinned against
  ``dft_direct``).
* ``mm_acc(A, B, C0, dtype, out)`` -- the accumulating form ``C0 + A*B``
  that the D functions of Sections 4.2 and 4.3 ask of the unit
  (X <- X + Y*Z); C0 holds stored output values ('f32', 'bf16' bits or
  'i32').  Rectangular shapes (Corollary 1) need nothing new: ``mm`` takes
  any (R x K) times (K x J).

Every function here is pinned by tests/test_oracle_pins.py against values the
mathematics fixes (exact rational brute force, closed forms, library
routines on special cases); none is "parity unpinned".
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_DTYPES = {"f16": 0, "bf16": 1, "i8": 2}
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_f16_to_f64.restype = ctypes.c_double
    lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_f64.restype = ctypes.c_double
    lib.oracle_f64_to_bf16_rne.argtypes = [ctypes.c_double]
    lib.oracle_f64_to_bf16_rne.restype = ctypes.c_uint16
    lib.oracle_f64_to_bf16_array.argtypes = [vp, vp, i64]
    lib.oracle_f64_to_bf16_array.restype = None
    lib.oracle_decode_array.argtypes = [ctypes.c_int, vp, vp, i64]
    lib.oracle_decode_array.restype = None
    lib.oracle_mm_f64.argtypes = [ctypes.c_int, vp, vp, i64, i64, i64, vp, i64, vp]
    lib.oracle_mm_f64.restype = ctypes.c_int
    lib.oracle_mm_i64.argtypes = [vp, vp, i64, i64, i64, vp, i64, vp]
    lib.oracle_mm_i64.restype = ctypes.c_int
    lib.oracle_poly_eval.argtypes = [ctypes.c_int, vp, i64, vp, i64, vp, vp]
    lib.oracle_poly_eval.restype = ctypes.c_int
    lib.oracle_transitive_closure.argtypes = [vp, i64, vp]
    lib.oracle_transitive_closure.restype = ctypes.c_int
    lib.oracle_dft_direct.argtypes = [vp, i64, i64, vp]
    lib.oracle_dft_direct.restype = ctypes.c_int
    lib.oracle_dft_direct_at.argtypes = [vp, i64, i64, vp, i64, vp]
    lib.oracle_dft_direct_at.restype = ctypes.c_int
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().oracle_threads())


def decode(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored f16/bf16 bit patterns (uint16) or int8 values to float64."""
    code = _DTYPES[dtype]
    want = np.int8 if dtype == "i8" else np.uint16
    bits = np.ascontiguousarray(bits).view(want)
    out = np.empty(bits.shape, dtype=np.float64)
    _load().oracle_decode_array(code, _ptr(bits), _ptr(out), bits.size)
    return out


def f16_to_f64(bits: np.ndarray) -> np.ndarray:
    return decode(bits, "f16")


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return decode(bits, "bf16")


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (RNE, one step); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_f64_to_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


def mm(A: np.ndarray, B: np.ndarray, dtype: str, rows=None) -> np.ndarray:
    """C = A*B (selected rows of it) as float64, or int64 for dtype 'i8'.

    A: (R, K) and B: (K, J) arrays of stored values: uint16 bit patterns for
    'f16'/'bf16' (int16 views are accepted), int8 for 'i8'.
    """
    if A.ndim != 2 or B.ndim != 2 or A.shape[1] != B.shape[0]:
        raise ValueError(f"shape mismatch: {A.shape} x {B.shape}")
    R, K = A.shape
    J = B.shape[1]
    lib = _load()
    if rows is None:
        ids_ptr, n_ids = None, R
    else:
        ids = np.ascontiguousarray(rows, dtype=np.int64)
        ids_ptr, n_ids = _ptr(ids), ids.size
    if dtype == "i8":
        a = np.ascontiguousarray(A).view(np.int8)
        b = np.ascontiguousarray(B).view(np.int8)
        out = np.empty((n_ids, J), dtype=np.int64)
        rc = lib.oracle_mm_i64(_ptr(a), _ptr(b), R, K, J, ids_ptr, n_ids, _ptr(out))
    else:
        a = np.ascontiguousarray(A).view(np.uint16)
        b = np.ascontiguousarray(B).view(np.uint16)
        out = np.empty((n_ids, J), dtype=np.float64)
        rc = lib.oracle_mm_f64(_DTYPES[dtype], _ptr(a), _ptr(b), R, K, J,
                               ids_ptr, n_ids, _ptr(out))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def decode_out(C0: np.ndarray, out: str) -> np.ndarray:
    """Stored output values as float64 (or int64 for 'i32')."""
    if out == "i32":
        return np.asarray(C0, dtype=np.int32).astype(np.int64)
    if out == "bf16":
        return bf16_to_f64(np.ascontiguousarray(C0).view(np.uint16))
    return np.asarray(C0, dtype=np.float32).astype(np.float64)


def mm_acc(A: np.ndarray, B: np.ndarray, C0: np.ndarray, dtype: str, out: str,
           rows=None) -> np.ndarray:
    """C0 + A*B for the selected rows, summed exactly in binary64 (or int64);
    the caller rounds once to the output format."""
    prod = mm(A, B, dtype, rows=rows)
    c0 = decode_out(C0, out)
    if rows is not None:
        c0 = c0[np.asarray(rows, dtype=np.int64)]
    return c0 + prod


def poly_eval(coef: np.ndarray, points: np.ndarray, dtype: str):
    """(values, magnitudes): A(x_i) = sum_h a_h x_i^h and sum_h |a_h| |x_i|^h
    for every point, from the stored 16-bit coefficients and points."""
    if dtype not in ("f16", "bf16"):
        raise ValueError("polynomial evaluation takes f16 or bf16 inputs")
    a = np.ascontiguousarray(coef).view(np.uint16).ravel()
    x = np.ascontiguousarray(points).view(np.uint16).ravel()
    val = np.empty(x.size, dtype=np.float64)
    mag = np.empty(x.size, dtype=np.float64)
    rc = _load().oracle_poly_eval(_DTYPES[dtype], _ptr(a), a.size, _ptr(x), x.size,
                                  _ptr(val), _ptr(mag))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return val, mag


def transitive_closure(d: np.ndarray) -> np.ndarray:
    """Closure of the n x n adjacency matrix d (nonzero = edge) as uint8 0/1."""
    d = np.ascontiguousarray(d).view(np.uint8)
    if d.ndim != 2 or d.shape[0] != d.shape[1]:
        raise ValueError("adjacency matrix must be square")
    out = np.empty_like(d)
    rc = _load().oracle_transitive_closure(_ptr(d), d.shape[0], _ptr(out))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out


def dft_direct(x: np.ndarray) -> np.ndarray:
    """DFT of every row of x (complex, shape (batch, n) or (n,)) by the
    definition, in binary64; returns complex128 of the same shape."""
    x = np.asarray(x, dtype=np.complex128)
    shape = x.shape
    x2 = np.ascontiguousarray(x.reshape(-1, shape[-1]))
    y = np.empty_like(x2)
    rc = _load().oracle_dft_direct(_ptr(x2.view(np.float64)), x2.shape[1], x2.shape[0],
                                   _ptr(y.view(np.float64)))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return y.reshape(shape)


def dft_direct_at(x: np.ndarray, ks) -> np.ndarray:
    """The definition y[k] = sum_j x[j] exp(-2 pi i j k / n) at the output
    frequencies ks only (binary64, O(n) per frequency), for every row of x
    (complex, shape (batch, n) or (n,)); returns complex128 of shape
    (batch, len(ks)) (or (len(ks),))."""
    x = np.asarray(x, dtype=np.complex128)
    one = x.ndim == 1
    x2 = np.ascontiguousarray(x.reshape(-1, x.shape[-1]))
    k = np.ascontiguousarray(ks, dtype=np.int64).ravel()
    y = np.empty((x2.shape[0], k.size), dtype=np.complex128)
    rc = _load().oracle_dft_direct_at(_ptr(x2.view(np.float64)), x2.shape[1], x2.shape[0],
                                      _ptr(k), k.size, _ptr(y.view(np.float64)))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return y[0] if one else y


def dft(x: np.ndarray) -> np.ndarray:
    """DFT of every row of x (complex) in binary64 through numpy's FFT."""
    return np.fft.fft(np.asarray(x, dtype=np.complex128), axis=-1)
