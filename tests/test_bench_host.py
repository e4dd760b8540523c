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
    # DFT: the 4 radix-32 levels of 2^20 run as 2 launches (levels 1-2 and
    # 3-4 fused), each reading and writing the array once
    w, b = bench.algorithmic(inputs.DFT_WORKLOADS["dft_c64_n1048576_b16_s32"])
    assert b == 2 * 2 * 8 * 16 * (1 << 20) and w == 5 * 16 * (1 << 20) * 20


@pytest.mark.parametrize("n,s,levels", [(1, 32, 1), (32, 32, 1), (64, 32, 2), (1024, 32, 2),
                                        (2048, 32, 3), (1 << 20, 32, 4), (1 << 20, 16, 5),
                                        (16, 16, 1), (1 << 30, 32, 6)])
def test_dft_levels(n, s, levels):
    assert bench.dft_levels(n, s) == levels


@pytest.mark.parametrize("n,s,launches", [(32, 32, 1), (1024, 32, 2), (1 << 14, 32, 2),
                                          (1 << 15, 32, 2), (1 << 20, 32, 2), (1 << 12, 16, 2),
                                          (1 << 16, 16, 2), (1 << 20, 16, 3), (2048, 16, 3)])
def test_dft_launches(n, s, launches):
    """Pairs of full-radix levels share a launch where the library fuses them
    (the pair conditions of the DFT launcher)."""
    assert bench.dft_launches(n, s) == launches


def test_multi_gpu_request_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_model_time_is_theorem2_form():
    """T = a * work + calls * l with the fit of the workload's types and unit
    size: for the product, a N^3/s + (N/s)^2 l."""
    fits = {"bf16_f32_s32": {"a_s_per_work": 2e-12, "ell_us": 4.0}}
    sp = inputs.WORKLOADS["gemm_bf16_N8192_s32"]
    N, s = 8192, 32
    mt = bench.model_time(sp, (N // s) ** 2, N ** 3 // s, 0.8, fits)
    want = 2e-12 * N ** 3 / s + (N // s) ** 2 * 4e-6
    assert abs(mt["T_model_ms"] - want * 1e3) <= 1e-9 * want * 1e3
    assert abs(mt["measured_over_model"] - 0.8e-3 / want) < 1e-12
    assert bench.model_time(inputs.WORKLOADS["gemm_i8_N8192_s32"], 1, 1, 1.0, fits) is None


class _FakeWorkload:
    """A measured workload whose 'GPU result' is the oracle's own, rounded to
    the output type: the baseline's sampling and parity logic must accept it."""

    def __init__(self, name, perturb=0.0):
        import numpy as np
        import torch
        import oracle
        self.spec = dict(inputs.WORKLOADS[name])
        self.A, self.B = inputs.make_inputs(self.spec)
        ref = oracle.mm(inputs.bits(self.A), inputs.bits(self.B), self.spec["dtype"])
        if self.spec["out"] == "i32":
            self.C = torch.from_numpy(ref.astype(np.int32))
        elif self.spec["out"] == "bf16":
            self.C = torch.from_numpy(oracle.f64_to_bf16(ref).view(np.int16)).view(torch.bfloat16)
        else:
            self.C = torch.from_numpy((ref * (1 + perturb)).astype(np.float32))


@pytest.mark.parametrize("name", ["tall_f16_n4096_s16", "gemm_f16_N1024_s16"])
def test_cpu_baseline_logic(name):
    rep = bench.cpu_baseline(_FakeWorkload(name), target_s=2.0)
    assert rep["kind"] == "oracle" and rep["cores"] >= 1 and rep["seconds"] > 0
    assert "output rows" in rep["sample"]


def test_cpu_baseline_rejects_a_wrong_result():
    with pytest.raises(AssertionError):
        bench.cpu_baseline(_FakeWorkload("gemm_f16_N1024_s16", perturb=0.01), target_s=2.0)


def test_host_info_fields():
    h = bench.host_info()
    assert {"cpu_model", "nproc", "OMP_NUM_THREADS", "oracle_threads"} <= set(h)
    assert h["nproc"] >= 1 and h["oracle_threads"] >= 1


def test_counted_traffic_reads_the_summaries():
    """Every counter summary under profiles/ parses; the bench takes its traffic
    only from one taken on the current kernel source, and for a call made of
    several launches (the closure) the per-call total."""
    import glob
    import os
    import re
    kinds = {"gemm": "gemm", "tall": "tall", "cor1": "rect", "pad": "rect", "poly": "poly",
             "tc": "tc", "dft": "dft"}
    paths = sorted(glob.glob(os.path.join(bench.PROFILES, "*_counters.txt")))
    assert paths
    for path in paths:
        name = os.path.basename(path)[:-len("_counters.txt")]
        kind = kinds[name.split("_")[0]]
        text = open(path).read()
        digest = re.search(r"^kernel_source_sha256: (\S+)", text, re.M).group(1)
        got = bench.counted_traffic(name, kind)
        if digest != bench.kernel_hash(kind):
            assert got is None
            continue
        per_call = re.search(r"^hbm_bytes_per_call: (\S+)", text, re.M)
        want = per_call or re.search(r"^hbm_bytes_per_dispatch: (\S+)", text, re.M)
        assert got == float(want.group(1))
        assert got > 0
