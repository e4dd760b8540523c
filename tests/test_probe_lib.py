"""The measurement probes of bench.py (libtcu_probe.so, not part of the C ABI
in include/tcu.h): without a GPU, the library loads, exports its five entry
points and rejects bad arguments before any HIP call; on the GPU, every probe
runs to completion on a small grid (the rates themselves are measured by
`bench.py --mfma-probe`)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_1908_06649_amd import build as hip_build
from paper_1908_06649_amd import tcu

PROBES = ("tcu_probe_mfma", "tcu_probe_overlap", "tcu_probe_lds", "tcu_probe_dma",
          "tcu_probe_pingpong")
FAKE = 0x10000000   # never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def P():
    if not os.path.exists(hip_build.PROBE_LIB):
        pytest.skip("libtcu_probe.so not built")
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    v, i64 = ctypes.c_void_p, ctypes.c_int64
    sig = {"tcu_probe_mfma": [ctypes.c_int, v, v, i64, ctypes.c_int, v],
           "tcu_probe_overlap": [ctypes.c_int, ctypes.c_int, v, v, i64, ctypes.c_int, v],
           "tcu_probe_lds": [ctypes.c_int, v, i64, ctypes.c_int, ctypes.c_int, v],
           "tcu_probe_dma": [v, v, i64, ctypes.c_int, ctypes.c_int, v],
           "tcu_probe_pingpong": [ctypes.c_int, v, v, v, i64, ctypes.c_int, v]}
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.restype = ctypes.c_int
        fn.argtypes = args
    return lib


def test_probe_library_exports(P):
    out = subprocess.run(["nm", "-D", "--defined-only", hip_build.PROBE_LIB],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (tcu_probe_[a-z0-9_]+)$", out, flags=re.M))
    assert set(PROBES) <= exported


def test_probe_bad_arguments_rejected(P):
    assert P.tcu_probe_mfma(0, None, FAKE, 1, 1, None) == -1
    assert P.tcu_probe_mfma(0, FAKE, FAKE, 0, 1, None) == -1
    assert P.tcu_probe_overlap(4, 0, FAKE, FAKE, 1, 1, None) == -1
    assert P.tcu_probe_overlap(0, 0, FAKE, FAKE, 1, 0, None) == -1
    assert P.tcu_probe_lds(0, FAKE, 1, 1, 384, None) == -1
    assert P.tcu_probe_lds(0, None, 1, 1, 256, None) == -1
    assert P.tcu_probe_lds(3, FAKE, 1, 1, 256, None) == -1
    assert P.tcu_probe_dma(None, FAKE, 1, 1, 256, None) == -1
    assert P.tcu_probe_dma(FAKE, FAKE, 1, 1, 128, None) == -1
    assert P.tcu_probe_dma(FAKE, FAKE, 0, 1, 256, None) == -1
    assert P.tcu_probe_pingpong(5, FAKE, FAKE, FAKE, 1, 1, None) == -1
    assert P.tcu_probe_pingpong(-1, FAKE, FAKE, FAKE, 1, 1, None) == -1
    assert P.tcu_probe_pingpong(0, FAKE, None, FAKE, 1, 1, None) == -1


@pytest.mark.gpu
def test_probes_run(P):
    import torch
    blocks = 4
    st = torch.cuda.current_stream()
    # operand words: mfma 12 x 16 B per lane (the largest), overlap 3 x 16 B per lane,
    # pingpong 2048 x 16 B per block
    ops = torch.randn(blocks * 512 * 12 * 8, device="cuda").to(torch.bfloat16).view(torch.int32)
    src = torch.zeros(1 << 18, dtype=torch.int32, device="cuda")          # 1 MiB
    out = torch.zeros(blocks * 1024, dtype=torch.int32, device="cuda")
    assert ops.numel() * 4 == blocks * 512 * 12 * 16 >= blocks * 2048 * 16
    s = st.cuda_stream
    for dt in (tcu.TCU_BF16_F32, tcu.TCU_I8_I32):
        assert P.tcu_probe_mfma(dt, ops.data_ptr(), out.data_ptr(), 2, blocks, s) == 0
    for mode in range(4):
        assert P.tcu_probe_overlap(mode, 2, ops.data_ptr(), out.data_ptr(), 2, blocks, s) == 0
    for kind in (0, 1, 2):
        for threads in (256, 512, 1024):
            assert P.tcu_probe_lds(kind, out.data_ptr(), 2, blocks, threads, s) == 0
    for threads in (256, 512, 1024):
        assert P.tcu_probe_dma(src.data_ptr(), out.data_ptr(), 2, blocks, threads, s) == 0
    for mode in range(5):
        assert P.tcu_probe_pingpong(mode, ops.data_ptr(), src.data_ptr(), out.data_ptr(), 3,
                                    blocks, s) == 0
    torch.cuda.synchronize()
