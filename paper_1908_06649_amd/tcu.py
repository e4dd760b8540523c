"""Python binding of the C ABI in include/tcu.h (argument marshalling only).

Functions carry the C names.  Matrices are torch tensors on the current HIP
device; torch supplies device memory and the stream, nothing else -- every
step of the computation runs in the library's HIP kernels.  There is no
fallback: if ``libtcu.so`` is missing or fails to load, every call raises.

    tcu_mm_tall(A, n, s, B, C)   C (n x s) = A (n x s) @ B (s x s)     (native call)
    tcu_gemm(A, B, C, N)         C (N x N) = A @ B, unit size tcu_get_unit()
    tcu_transitive_closure(X, n, ld)   X <- transitive closure, in place (Theorem 5)
    tcu_dft(x, y, work, n, batch)   y[b] = DFT(x[b]), complex64        (Theorem 7)
    tcu_poly_eval(coef, n, points, p, out)
                                 out[i] = sum_h coef[h] * points[i]**h    (Theorem 11)
    tcu_gemm_rect(A, lda, B, ldb, C, ldc, M, K, N, flags)
                                 C (M x N) = [C +] A (M x K) @ B (K x N); A, B and C
                                 may be row-strided 2-D views (row pitch = ld)

The element types are taken from the tensors: (float16 -> float32),
(bfloat16 -> float32), (bfloat16 -> bfloat16) or (int8 -> int32).  Calls are
issued on torch's current stream and are asynchronous.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtcu.so")

TCU_OK = 0
TCU_ERR_NULL = -1
TCU_ERR_SHAPE = -2
TCU_ERR_UNSUPPORTED = -3
TCU_ERR_ALIGN = -4
TCU_ERR_OVERLAP = -5
TCU_ERR_HIP = -6
TCU_ERR_NO_DEVICE = -7
TCU_ERR_POINTER = -8
TCU_ERR_SCRATCH = -9

TCU_F16_F32 = 0
TCU_BF16_F32 = 1
TCU_BF16_BF16 = 2
TCU_I8_I32 = 3

TCU_ACCUMULATE = 1

# Test overrides and the pointer-check switch (tcu_set_knob)
TCU_KNOB_GEMM_KERNEL = 0
TCU_KNOB_PP_GRID = 1
TCU_KNOB_SPLIT_K = 2
TCU_KNOB_TAIL_SPLIT = 3
TCU_KNOB_CHECK_POINTERS = 4
TCU_KNOB_DFT_PAIRS = 5
TCU_PATH_AUTO = 0
TCU_PATH_FULL_TILE = 1
TCU_PATH_GENERAL = 2
TCU_PATH_RING = 3
TCU_MAX_RECT_DIM = 1 << 30

# Every symbol include/tcu.h declares: name -> (restype, argtypes)
_i64, _int, _vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
SIGNATURES = {
    "tcu_set_unit": (_int, [_int]),
    "tcu_get_unit": (_int, []),
    "tcu_set_dtype": (_int, [_int]),
    "tcu_get_dtype": (_int, []),
    "tcu_set_stream": (_int, [_vp]),
    "tcu_get_stream": (_vp, []),
    "tcu_mm_tall": (_int, [_vp, _i64, _int, _vp, _vp]),
    "tcu_gemm": (_int, [_vp, _vp, _vp, _i64]),
    "tcu_mm_tall_ex": (_int, [_vp, _i64, _int, _vp, _vp, _int, _vp]),
    "tcu_gemm_ex": (_int, [_vp, _vp, _vp, _i64, _int, _int, _vp]),
    "tcu_gemm_rect": (_int, [_vp, _i64, _vp, _i64, _vp, _i64, _i64, _i64, _i64, _int]),
    "tcu_gemm_rect_ex": (_int, [_vp, _i64, _vp, _i64, _vp, _i64, _i64, _i64, _i64, _int,
                                _int, _int, _vp]),
    "tcu_poly_eval": (_int, [_vp, _i64, _vp, _i64, _vp]),
    "tcu_poly_eval_ex": (_int, [_vp, _i64, _vp, _i64, _vp, _int, _int, _vp]),
    "tcu_transitive_closure": (_int, [_vp, _i64, _i64]),
    "tcu_transitive_closure_ex": (_int, [_vp, _i64, _i64, _int, _vp]),
    "tcu_dft": (_int, [_vp, _vp, _vp, _i64, _i64]),
    "tcu_dft_ex": (_int, [_vp, _vp, _vp, _i64, _i64, _int, _vp]),
    "tcu_dft_noalloc": (_int, [_vp, _vp, _i64, _i64, _int, _vp]),
    "tcu_calls": (_i64, []),
    "tcu_square_calls": (_i64, []),
    "tcu_work": (_i64, []),
    "tcu_reset_calls": (None, []),
    "tcu_strerror": (ctypes.c_char_p, [_int]),
    "tcu_check_device_range": (_int, [_vp, _i64]),
    "tcu_set_knob": (_int, [_int, _int]),
    "tcu_get_knob": (_int, [_int]),
}

_lib = None


class TcuError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {tcu_strerror(status)} (status {status})")


def lib() -> ctypes.CDLL:
    """The loaded C library (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build the HIP library first "
                "(python -c 'import __graft_entry__ as g; g.build()')")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(rc: int, where: str) -> None:
    if rc != TCU_OK:
        raise TcuError(rc, where)


_DTYPES = None


def _dtype_code(a_dtype, c_dtype) -> int:
    global _DTYPES
    if _DTYPES is None:
        import torch
        _DTYPES = {
            (torch.float16, torch.float32): TCU_F16_F32,
            (torch.bfloat16, torch.float32): TCU_BF16_F32,
            (torch.bfloat16, torch.bfloat16): TCU_BF16_BF16,
            (torch.int8, torch.int32): TCU_I8_I32,
        }
    code = _DTYPES.get((a_dtype, c_dtype))
    if code is None:
        raise TcuError(TCU_ERR_UNSUPPORTED, f"dtype pair ({a_dtype}, {c_dtype})")
    return code


def _check_current_device(where: str, dev: int) -> None:
    """The library launches on the current HIP device: the tensors must be
    there (select it with torch.cuda.device(...))."""
    import torch
    cur = torch.cuda.current_device()
    if dev != cur:
        raise ValueError(f"{where}: tensors are on cuda:{dev}, the current device is cuda:{cur}")


def _marshal(where: str, tensors, numels):
    """Check that tensors are contiguous, on one HIP device (the current one),
    and sized as the call will read/write them; return the device index and
    their device pointers."""
    dev = tensors[0].get_device() if tensors[0].is_cuda else -1
    ptrs = []
    for t, want in zip(tensors, numels):
        if not t.is_cuda or t.get_device() != dev:
            raise ValueError(f"{where}: all matrices must be on the same HIP device")
        if not t.is_contiguous():
            raise ValueError(f"{where}: matrices must be contiguous (row-major)")
        if t.numel() != want:
            raise ValueError(f"{where}: expected {want} elements, got {t.numel()}")
        ptrs.append(t.data_ptr())
    _check_current_device(where, dev)
    return dev, ptrs


_RAW_STREAM = None


def _stream_ptr(dev: int) -> int:
    """The current torch stream of device dev, as a hipStream_t value."""
    global _RAW_STREAM
    if _RAW_STREAM is None:
        import torch
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        _RAW_STREAM = raw if raw is not None else (
            lambda d: torch.cuda.current_stream(d).cuda_stream)
    return _RAW_STREAM(dev)


# ------------------------------------------------------------ configuration
def tcu_set_unit(s: int) -> None:
    _check(lib().tcu_set_unit(int(s)), "tcu_set_unit")


def tcu_get_unit() -> int:
    return int(lib().tcu_get_unit())


def tcu_set_dtype(dtype: int) -> None:
    _check(lib().tcu_set_dtype(int(dtype)), "tcu_set_dtype")


def tcu_get_dtype() -> int:
    return int(lib().tcu_get_dtype())


def tcu_set_stream(stream_ptr: int | None) -> None:
    _check(lib().tcu_set_stream(stream_ptr), "tcu_set_stream")


def tcu_get_stream() -> int | None:
    return lib().tcu_get_stream()


# ------------------------------------------------------------------- calls
def tcu_mm_tall(A, n: int, s: int, B, C) -> None:
    """Native call: C (n x s) = A (n x s) @ B (s x s); s must equal the unit size."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal("tcu_mm_tall", (A, B, C), (n * s, s * s, n * s))
    L = lib()
    _check(L.tcu_set_dtype(dt), "tcu_mm_tall")
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_mm_tall")
    _check(L.tcu_mm_tall(pa, int(n), int(s), pb, pc), "tcu_mm_tall")


def tcu_gemm(A, B, C, N: int) -> None:
    """Blocked product of Theorem 2: C (N x N) = A @ B with unit size tcu_get_unit()."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal("tcu_gemm", (A, B, C), (N * N, N * N, N * N))
    L = lib()
    _check(L.tcu_set_dtype(dt), "tcu_gemm")
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_gemm")
    _check(L.tcu_gemm(pa, pb, pc, int(N)), "tcu_gemm")


def tcu_mm_tall_ex(A, n: int, s: int, B, C, stream_ptr: int | None = None) -> None:
    """Stateless native call (unit size, dtype and stream as arguments)."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal("tcu_mm_tall_ex", (A, B, C), (n * s, s * s, n * s))
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_mm_tall_ex(pa, int(n), int(s), pb, pc, dt, st), "tcu_mm_tall_ex")


def tcu_gemm_ex(A, B, C, N: int, s: int, stream_ptr: int | None = None) -> None:
    """Stateless blocked product (unit size, dtype and stream as arguments)."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal("tcu_gemm_ex", (A, B, C), (N * N, N * N, N * N))
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_gemm_ex(pa, pb, pc, int(N), int(s), dt, st), "tcu_gemm_ex")


def _marshal_views(where: str, views):
    """(tensor, rows, cols, ld) per operand: check that each is a 2-D view of
    that shape with unit column stride and row pitch ld on one HIP device
    (the current one); return the device index and the view base pointers."""
    dev = views[0][0].get_device() if views[0][0].is_cuda else -1
    ptrs = []
    for t, rows, cols, ld in views:
        if not t.is_cuda or t.get_device() != dev:
            raise ValueError(f"{where}: all matrices must be on the same HIP device")
        if t.dim() != 2 or tuple(t.shape) != (rows, cols):
            raise ValueError(f"{where}: expected a {rows} x {cols} view, got {tuple(t.shape)}")
        if cols > 1 and t.stride(1) != 1:
            raise ValueError(f"{where}: rows must be contiguous (column stride 1)")
        if rows > 1 and t.stride(0) != ld:
            raise ValueError(f"{where}: row pitch {t.stride(0)} does not match ld={ld}")
        ptrs.append(t.data_ptr())
    _check_current_device(where, dev)
    return dev, ptrs


def tcu_gemm_rect(A, lda: int, B, ldb: int, C, ldc: int, M: int, K: int, N: int,
                  flags: int = 0) -> None:
    """C (M x N) = A (M x K) @ B (K x N), or C += A @ B with flags=TCU_ACCUMULATE
    (Corollary 1 / the D functions' update); unit size tcu_get_unit()."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal_views(
        "tcu_gemm_rect", ((A, M, K, lda), (B, K, N, ldb), (C, M, N, ldc)))
    L = lib()
    _check(L.tcu_set_dtype(dt), "tcu_gemm_rect")
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_gemm_rect")
    _check(L.tcu_gemm_rect(pa, int(lda), pb, int(ldb), pc, int(ldc), int(M), int(K), int(N),
                           int(flags)), "tcu_gemm_rect")


def tcu_gemm_rect_ex(A, lda: int, B, ldb: int, C, ldc: int, M: int, K: int, N: int, flags: int,
                     s: int, stream_ptr: int | None = None) -> None:
    """Stateless rectangular / accumulating product (unit size, dtype, stream as arguments)."""
    dt = _dtype_code(A.dtype, C.dtype)
    dev, (pa, pb, pc) = _marshal_views(
        "tcu_gemm_rect_ex", ((A, M, K, lda), (B, K, N, ldb), (C, M, N, ldc)))
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_gemm_rect_ex(pa, int(lda), pb, int(ldb), pc, int(ldc), int(M), int(K),
                                  int(N), int(flags), int(s), dt, st), "tcu_gemm_rect_ex")


def _poly_dtype(pts_dtype, out_dtype) -> int:
    import torch
    table = {(torch.float16, torch.float32): TCU_F16_F32,
             (torch.bfloat16, torch.float32): TCU_BF16_F32,
             (torch.bfloat16, torch.bfloat16): TCU_BF16_BF16}
    try:
        return table[(pts_dtype, out_dtype)]
    except KeyError:
        raise TcuError(TCU_ERR_UNSUPPORTED, f"dtype pair ({pts_dtype}, {out_dtype})") from None


def tcu_poly_eval(coef, n: int, points, p: int, out) -> None:
    """Theorem 11: out[i] = sum_{h<n} coef[h] * points[i]**h, unit size tcu_get_unit()."""
    dt = _poly_dtype(points.dtype, out.dtype)
    if coef.dtype != points.dtype:
        raise ValueError("tcu_poly_eval: coefficients and points must share one input type")
    dev, (ppts, pcoef, pout) = _marshal("tcu_poly_eval", (points, coef, out), (p, n, p))
    L = lib()
    _check(L.tcu_set_dtype(dt), "tcu_poly_eval")
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_poly_eval")
    _check(L.tcu_poly_eval(pcoef or None, int(n), ppts or None, int(p), pout or None),
           "tcu_poly_eval")


def tcu_poly_eval_ex(coef, n: int, points, p: int, out, s: int,
                     stream_ptr: int | None = None) -> None:
    """Stateless batch polynomial evaluation (unit size, dtype, stream as arguments)."""
    dt = _poly_dtype(points.dtype, out.dtype)
    if coef.dtype != points.dtype:
        raise ValueError("tcu_poly_eval_ex: coefficients and points must share one input type")
    dev, (ppts, pcoef, pout) = _marshal("tcu_poly_eval_ex", (points, coef, out), (p, n, p))
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_poly_eval_ex(pcoef or None, int(n), ppts or None, int(p), pout or None,
                                  int(s), dt, st), "tcu_poly_eval_ex")


def tcu_transitive_closure(X, n: int, ld: int) -> None:
    """Theorem 5, in place: X (an n x n int8 view with row pitch ld) becomes
    the transitive closure of the graph it is the adjacency matrix of."""
    import torch
    if X.dtype not in (torch.int8, torch.uint8):
        raise ValueError("tcu_transitive_closure: X must be int8 or uint8")
    dev, (px,) = _marshal_views("tcu_transitive_closure", ((X, n, n, ld),))
    L = lib()
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_transitive_closure")
    _check(L.tcu_transitive_closure(px or None, int(n), int(ld)), "tcu_transitive_closure")


def tcu_transitive_closure_ex(X, n: int, ld: int, s: int, stream_ptr: int | None = None) -> None:
    """Stateless transitive closure (unit size and stream as arguments)."""
    import torch
    if X.dtype not in (torch.int8, torch.uint8):
        raise ValueError("tcu_transitive_closure_ex: X must be int8 or uint8")
    dev, (px,) = _marshal_views("tcu_transitive_closure_ex", ((X, n, n, ld),))
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_transitive_closure_ex(px or None, int(n), int(ld), int(s), st),
           "tcu_transitive_closure_ex")


def _dft_args(where, x, y, work, n, batch):
    import torch
    for name, t in (("x", x), ("y", y)):
        if t.dtype != torch.complex64:
            raise ValueError(f"{where}: {name} must be complex64")
    tensors = [x, y] + ([work] if work is not None else [])
    dev, ptrs = _marshal(where, tensors, [n * batch] * len(tensors))
    if work is not None and work.dtype != torch.complex64:
        raise ValueError(f"{where}: work must be complex64")
    pw = ptrs[2] if work is not None else None
    return dev, (ptrs[0] or None), (ptrs[1] or None), (pw or None)


def tcu_dft(x, y, work, n: int, batch: int) -> None:
    """Theorem 7: y[b] = DFT(x[b]) for b < batch (complex64 tensors of
    batch * n elements); work is scratch of the same size (None if n <= s)."""
    dev, px, py, pw = _dft_args("tcu_dft", x, y, work, n, batch)
    L = lib()
    _check(L.tcu_set_stream(_stream_ptr(dev)), "tcu_dft")
    _check(L.tcu_dft(px, py, pw, int(n), int(batch)), "tcu_dft")


def tcu_dft_ex(x, y, work, n: int, batch: int, s: int, stream_ptr: int | None = None) -> None:
    """Stateless DFT (unit size and stream as arguments)."""
    dev, px, py, pw = _dft_args("tcu_dft_ex", x, y, work, n, batch)
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_dft_ex(px, py, pw, int(n), int(batch), int(s), st), "tcu_dft_ex")


TCU_DFT_NOALLOC_MAX_BYTES = 64 << 20


def tcu_dft_noalloc(x, y, n: int, batch: int, s: int, stream_ptr: int | None = None) -> None:
    """The DFT with the levels' second buffer in the library's fixed device
    scratch (no allocation; batch * n * 8 <= TCU_DFT_NOALLOC_MAX_BYTES when
    n > s); calls overlapping in time on one device race on that scratch."""
    dev, px, py, _ = _dft_args("tcu_dft_noalloc", x, y, None, n, batch)
    st = _stream_ptr(dev) if stream_ptr is None else stream_ptr
    _check(lib().tcu_dft_noalloc(px, py, int(n), int(batch), int(s), st), "tcu_dft_noalloc")


# --------------------------------------------------------- cost accounting
def tcu_calls() -> int:
    return int(lib().tcu_calls())


def tcu_square_calls() -> int:
    return int(lib().tcu_square_calls())


def tcu_work() -> int:
    return int(lib().tcu_work())


def tcu_reset_calls() -> None:
    lib().tcu_reset_calls()


def tcu_strerror(status: int) -> str:
    return lib().tcu_strerror(int(status)).decode()


# ------------------------------------------- pointer checks, test overrides
def tcu_check_device_range(ptr: int, nbytes: int) -> int:
    """Status of the pointer check for [ptr, ptr + nbytes) (TCU_OK or a
    negative code; returned, not raised)."""
    return int(lib().tcu_check_device_range(ptr or None, int(nbytes)))


def tcu_set_knob(knob: int, value: int) -> None:
    _check(lib().tcu_set_knob(int(knob), int(value)), "tcu_set_knob")


def tcu_get_knob(knob: int) -> int:
    return int(lib().tcu_get_knob(int(knob)))
