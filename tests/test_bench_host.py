"""Host logic of bench.py (CPU only): the algorithmic work and bytes it
divides by time, against the figures worked out for each workload from the
method's definitions, and the single-GPU contract."""
import os
import subprocess
import sys

import pytest

from paper_1908_06649_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

# (work, bytes) per call: 2 n s^2 flop and n s in + s^2 in + n s out bytes
# for the native call (Section 3); 2 N^3 flop and the operands and result
# once for the product (Theorem 2).
EXPECTED = {
    "tall_f16_n4096_s16": (2_097_152, 393_728),
    "gemm_f16_N1024_s16": (2_147_483_648, 8_388_608),
    "gemm_bf16_N8192_s32": (1_099_511_627_776, 536_870_912),
    "gemm_i8_N8192_s32": (1_099_511_627_776, 402_653_184),
    "tall_bf16_n16777216_s32": (34_359_738_368, 2_147_485_696),
}


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_algorithmic_work_and_bytes(name):
    work, nbytes = bench.algorithmic(inputs.WORKLOADS[name])
    assert (work, nbytes) == EXPECTED[name]


def test_algorithmic_rect_poly_tc_dft():
    # Corollary 1, accumulating: C is read and written
    M, K, N = 8192, 2048, 8192
    w, b = bench.algorithmic(inputs.RECT_WORKLOADS["cor1_bf16_M8192_K2048_N8192_acc"])
    assert w == 2 * M * K * N and b == (M * K + K * N) * 2 + 2 * M * N * 4
    # Theorem 11: 2 p n multiply-adds; coefficients, points and values once
    n, p = 4096, 1 << 24
    w, b = bench.algorithmic(inputs.POLY_WORKLOADS["poly_bf16_n4096_p16777216_s32"])
    assert w == 2 * n * p and b == 2 * n + 2 * p + 4 * p
    # one pivot band (n <= 256): the diagonal block read and written, plus
    # the normalizing pass
    w, b = bench.algorithmic({"kind": "tc", "n": 256})
    assert w == 2 * 256 ** 3 and b == 2 * 256 * 256 + 2 * 256 * 256
    # DFT: each of the 4 radix-32 levels of 2^20 reads and writes the array
    w, b = bench.algorithmic(inputs.DFT_WORKLOADS["dft_c64_n1048576_b16_s32"])
    assert b == 4 * 2 * 8 * 16 * (1 << 20) and w == 5 * 16 * (1 << 20) * 20


@pytest.mark.parametrize("n,s,levels", [(1, 32, 1), (32, 32, 1), (64, 32, 2), (1024, 32, 2),
                                        (2048, 32, 3), (1 << 20, 32, 4), (1 << 20, 16, 5),
                                        (16, 16, 1), (1 << 30, 32, 6)])
def test_dft_levels(n, s, levels):
    assert bench.dft_levels(n, s) == levels


def test_multi_gpu_request_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr
