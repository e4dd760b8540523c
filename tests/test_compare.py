"""The parity checker itself (CPU only): it accepts correct results and
rejects plausible wrong ones, so a GPU test cannot pass vacuously."""
import numpy as np
import pytest
import torch

import oracle
from oracle import compare
from paper_1908_06649_amd import inputs


def _case(dtype, n=64, K=32, J=32, seed=0):
    g = torch.Generator().manual_seed(seed)
    dist = "int8" if dtype == "i8" else "normal"
    A = inputs.bits(inputs.draw((n, K), dtype, dist, g))
    B = inputs.bits(inputs.draw((K, J), dtype, dist, g))
    return A, B, oracle.mm(A, B, dtype)


def test_float_accepts_binary32_rounding_and_rejects_errors():
    A, B, ref = _case("bf16")
    compare.check("bf16", "f32", A, B, ref.astype(np.float32))
    bad = ref.astype(np.float32).copy()
    bad[3, 4] += 0.05 * abs(bad[3, 4]) + 0.5
    with pytest.raises(AssertionError):
        compare.check("bf16", "f32", A, B, bad)
    with pytest.raises(AssertionError):
        compare.check("bf16", "f32", A, B, np.roll(ref, 1, axis=0).astype(np.float32))


def test_bf16_accepts_rne_and_binary32_then_rne():
    A, B, ref = _case("bf16", n=200, K=32)
    compare.check("bf16", "bf16", A, B, oracle.f64_to_bf16(ref))
    via32 = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16)
    compare.check("bf16", "bf16", A, B, via32.view(torch.int16).numpy().view(np.uint16))


def test_bf16_rejects_truncation():
    A, B, ref = _case("bf16", n=400, K=32, seed=3)
    f32 = ref.astype(np.float32)
    trunc = (f32.view(np.uint32) >> 16).astype(np.uint16)   # round toward zero
    with pytest.raises(AssertionError):
        compare.check("bf16", "bf16", A, B, trunc)


def test_int_exact():
    A, B, ref = _case("i8")
    compare.check("i8", "i32", A, B, ref.astype(np.int32))
    bad = ref.astype(np.int32).copy()
    bad[0, 0] += 1
    with pytest.raises(AssertionError):
        compare.check("i8", "i32", A, B, bad)
