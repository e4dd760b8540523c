"""Helpers for the GPU parity tests: run the library's calls on seeded inputs
and hand results back as numpy arrays in the form the oracle compares."""
import numpy as np
import torch

from paper_1908_06649_amd import inputs, tcu

OUT = {"f16": "f32", "bf16": "f32", "i8": "i32"}
DEV = "cuda"


def out_dtype(name):
    return inputs.TORCH_DTYPE[name]


def to_np(C: torch.Tensor) -> np.ndarray:
    C = C.cpu()
    if C.dtype == torch.bfloat16:
        return C.view(torch.int16).numpy().view(np.uint16)
    return C.numpy()


def sentinel_buffer(numel: int, dtype: torch.dtype, guard: int = 4096):
    """A device buffer with a guard region after the first `numel` elements,
    all filled with a recognisable pattern; returns (buffer, view-to-use)."""
    buf = torch.empty(numel + guard, dtype=dtype, device=DEV)
    if dtype.is_floating_point:
        buf.fill_(float("nan"))
    else:
        buf.fill_(-0x5A5A5A5A if dtype == torch.int32 else 0x5A)
    return buf, buf[:numel]


def guard_intact(buf: torch.Tensor, numel: int) -> bool:
    g = buf[numel:]
    if buf.dtype.is_floating_point:
        return bool(torch.isnan(g).all())
    return bool((g == (-0x5A5A5A5A if buf.dtype == torch.int32 else 0x5A)).all())


def run_tall(A: torch.Tensor, B: torch.Tensor, s: int, out: str, check_guard=True):
    n = A.shape[0]
    buf, C = sentinel_buffer(n * s, out_dtype(out))
    tcu.tcu_set_unit(s)
    tcu.tcu_mm_tall(A.to(DEV), n, s, B.to(DEV), C.view(n, s))
    torch.cuda.synchronize()
    if check_guard:
        assert guard_intact(buf, n * s), "tall call wrote past the end of C"
    return to_np(C.view(n, s))


def run_gemm(A: torch.Tensor, B: torch.Tensor, s: int, out: str, check_guard=True):
    N = A.shape[0]
    buf, C = sentinel_buffer(N * N, out_dtype(out))
    tcu.tcu_set_unit(s)
    tcu.tcu_gemm(A.to(DEV), B.to(DEV), C.view(N, N), N)
    torch.cuda.synchronize()
    if check_guard:
        assert guard_intact(buf, N * N), "product wrote past the end of C"
    return to_np(C.view(N, N))


def draw_pair(a_shape, b_shape, dtype, seed):
    dist = "int8" if dtype == "i8" else "normal"
    g = torch.Generator().manual_seed(seed)
    return inputs.draw(a_shape, dtype, dist, g), inputs.draw(b_shape, dtype, dist, g)


# ------------------------------------------------ rectangular / accumulate
NAN_BITS = {"f16": 0x7E00, "bf16": 0x7FC0}


def _pad_fill(dtype_name: str):
    """Fill value for the unused columns of a padded input array: NaN for
    floating point (a kernel that reads past the view then poisons its sums)
    and 127 for int8."""
    return NAN_BITS.get(dtype_name, 127)


def pitched_input(X: torch.Tensor, ld: int, dtype_name: str) -> torch.Tensor:
    """Copy host matrix X (rows x cols) into a device array of row pitch ld,
    the columns past cols poisoned; returns the rows x cols view."""
    rows, cols = X.shape
    buf = torch.empty(max(rows, 1), max(ld, 1), dtype=X.dtype, device=DEV)
    if X.dtype == torch.int8:
        buf.fill_(_pad_fill(dtype_name))
    else:
        buf.view(torch.int16).fill_(_pad_fill(dtype_name))
    view = buf[:rows, :cols]
    view.copy_(X.to(DEV))
    return view


def c0_draw(shape, out: str, seed: int) -> torch.Tensor:
    """A seeded initial output for the accumulating form (host tensor)."""
    g = torch.Generator().manual_seed(seed)
    if out == "i32":
        return torch.randint(-(1 << 20), 1 << 20, shape, generator=g, dtype=torch.int32)
    x = torch.randn(shape, generator=g, dtype=torch.float32)
    return x.to(torch.bfloat16) if out == "bf16" else x


OUT_SENTINEL = {torch.float32: float("nan"), torch.bfloat16: float("nan"),
                torch.int32: -0x5A5A5A5A}


def run_rect(A: torch.Tensor, B: torch.Tensor, s: int, in_name: str, out: str,
             lda: int, ldb: int, ldc: int, C0: torch.Tensor | None = None):
    """tcu_gemm_rect on pitched device copies; the call accumulates into C0
    when it is given.  Checks that nothing outside the M x N view of C (the
    rest of its rows and a guard region after the array) was written.
    Returns the result as numpy."""
    M, K = A.shape
    N = B.shape[1]
    dA = pitched_input(A, ld=lda, dtype_name=in_name)
    dB = pitched_input(B, ld=ldb, dtype_name=in_name)
    odt = out_dtype(out)
    rows = max(M, 1)
    total = rows * max(ldc, 1)
    buf, flat = sentinel_buffer(total, odt)
    C = flat.view(rows, max(ldc, 1))[:M, :N]
    if C0 is not None:
        C.copy_(C0.to(DEV))
    tcu.tcu_set_unit(s)
    tcu.tcu_gemm_rect(dA, lda, dB, ldb, C, ldc, M, K, N,
                      tcu.TCU_ACCUMULATE if C0 is not None else 0)
    torch.cuda.synchronize()
    outside = flat.view(rows, max(ldc, 1))[:, N:]
    sent = OUT_SENTINEL[odt]
    if odt.is_floating_point:
        assert bool(torch.isnan(outside.float()).all()), "wrote into C's row padding"
    else:
        assert bool((outside == sent).all()), "wrote into C's row padding"
    assert guard_intact(buf, total), "wrote past the end of C"
    return to_np(C.contiguous())


# Names of the product's kernel paths -> TCU_KNOB_GEMM_KERNEL values
PATHS = {"auto": tcu.TCU_PATH_AUTO, "fast": tcu.TCU_PATH_FULL_TILE,
         "general": tcu.TCU_PATH_GENERAL, "ring": tcu.TCU_PATH_RING}
