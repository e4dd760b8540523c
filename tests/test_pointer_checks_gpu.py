"""Pointer checks (TCU_KNOB_CHECK_POINTERS / TCU_DEBUG), through the C ABI.

First the check itself, with no launch: device tensors pass, host memory,
pinned host memory, NULL and ranges running past their allocation are
TCU_ERR_POINTER.  Only then, with the checks on, every entry point is called
with one host operand and must return TCU_ERR_POINTER before any launch,
leaving its output untouched and its call uncounted; and valid calls with
the checks on still compute the oracle's result."""

import numpy as np
import pytest
import torch

from oracle import compare
from paper_1908_06649_amd import inputs, tcu

import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture
def checks_on(knobs):
    knobs(tcu.TCU_KNOB_CHECK_POINTERS, 1)
    assert tcu.tcu_get_knob(tcu.TCU_KNOB_CHECK_POINTERS) == 1


def test_check_device_range_alone():
    L = tcu.lib()
    big = torch.empty(16 << 20, dtype=torch.uint8, device=gu.DEV)   # a segment of its own
    p = big.data_ptr()
    assert L.tcu_check_device_range(p, big.numel()) == tcu.TCU_OK
    assert L.tcu_check_device_range(p + 4096, 4096) == tcu.TCU_OK
    assert L.tcu_check_device_range(p, 1 << 40) == tcu.TCU_ERR_POINTER       # past the segment
    host = np.zeros(1 << 16, dtype=np.uint8)
    assert L.tcu_check_device_range(host.ctypes.data, host.nbytes) == tcu.TCU_ERR_POINTER
    pinned = torch.zeros(1 << 16, dtype=torch.uint8, pin_memory=True)
    assert L.tcu_check_device_range(pinned.data_ptr(), pinned.numel()) == tcu.TCU_ERR_POINTER
    assert L.tcu_check_device_range(None, 16) == tcu.TCU_ERR_POINTER
    assert L.tcu_check_device_range(None, 0) == tcu.TCU_OK
    # a failed query leaves no error behind for the next HIP call
    torch.cuda.synchronize()
    x = torch.ones(8, device=gu.DEV) * 2
    assert float(x.sum()) == 16.0


def test_entry_points_reject_host_operands(checks_on):
    L = tcu.lib()
    host = np.zeros(1 << 22, dtype=np.uint8)       # 4 MiB, 16-byte aligned by numpy
    assert host.ctypes.data % 16 == 0
    hp = host.ctypes.data
    assert L.tcu_check_device_range(hp, 1024) == tcu.TCU_ERR_POINTER
    s, n = 32, 1024
    dA = torch.zeros(n, s, dtype=torch.bfloat16, device=gu.DEV)
    dB = torch.zeros(s, s, dtype=torch.bfloat16, device=gu.DEV)
    C = torch.full((n, s), 3.0, dtype=torch.float32, device=gu.DEV)
    tcu.tcu_reset_calls()
    st = None
    assert L.tcu_mm_tall_ex(hp, n, s, dB.data_ptr(), C.data_ptr(), tcu.TCU_BF16_F32, st) == \
        tcu.TCU_ERR_POINTER
    assert L.tcu_mm_tall_ex(dA.data_ptr(), n, s, hp, C.data_ptr(), tcu.TCU_BF16_F32, st) == \
        tcu.TCU_ERR_POINTER
    assert L.tcu_mm_tall_ex(dA.data_ptr(), n, s, dB.data_ptr(), hp, tcu.TCU_BF16_F32, st) == \
        tcu.TCU_ERR_POINTER
    N = 256
    dM = torch.zeros(N, N, dtype=torch.bfloat16, device=gu.DEV)
    CM = torch.full((N, N), 3.0, dtype=torch.float32, device=gu.DEV)
    assert L.tcu_gemm_ex(dM.data_ptr(), hp, CM.data_ptr(), N, s, tcu.TCU_BF16_F32, st) == \
        tcu.TCU_ERR_POINTER
    assert L.tcu_gemm_rect_ex(hp, N, dM.data_ptr(), N, CM.data_ptr(), N, N, N, N, 0, s,
                              tcu.TCU_BF16_F32, st) == tcu.TCU_ERR_POINTER
    out = torch.full((1000,), 3.0, dtype=torch.float32, device=gu.DEV)
    pts = torch.zeros(1000, dtype=torch.bfloat16, device=gu.DEV)
    assert L.tcu_poly_eval_ex(hp, 100, pts.data_ptr(), 1000, out.data_ptr(), s,
                              tcu.TCU_BF16_F32, st) == tcu.TCU_ERR_POINTER
    assert L.tcu_transitive_closure_ex(hp, 300, 300, s, st) == tcu.TCU_ERR_POINTER
    y = torch.zeros(4096, dtype=torch.complex64, device=gu.DEV)
    w = torch.zeros(4096, dtype=torch.complex64, device=gu.DEV)
    assert L.tcu_dft_ex(hp, y.data_ptr(), w.data_ptr(), 4096, 1, s, st) == tcu.TCU_ERR_POINTER
    torch.cuda.synchronize()
    assert bool((C == 3.0).all()) and bool((CM == 3.0).all()) and bool((out == 3.0).all())
    assert tcu.tcu_calls() == 0


def test_valid_calls_with_checks_on(checks_on):
    A, B = gu.draw_pair((4096, 32), (32, 32), "bf16", seed=21)
    got = gu.run_tall(A, B, 32, "bf16")
    compare.check("bf16", "bf16", inputs.bits(A), inputs.bits(B), got)
    A, B = gu.draw_pair((512, 512), (512, 512), "i8", seed=22)
    got = gu.run_gemm(A, B, 32, "i32")
    compare.check("i8", "i32", inputs.bits(A), inputs.bits(B), got)
