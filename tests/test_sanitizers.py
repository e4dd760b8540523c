"""Sanitizer builds of the host code (CPU only): the C ABI's argument
validation (tcu_abi.cpp, built with g++ as host code and linked against the
library's kernel objects) and the CPU oracle (tcu_oracle.c), both with
AddressSanitizer and UndefinedBehaviorSanitizer, each driven by a small C
program under tests/sanitize/ that exercises rejected, boundary and empty
arguments.  Any out-of-bounds access, use after free, leak (oracle), signed
overflow or other undefined behaviour aborts the driver."""
import os
import shutil
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-g", "-O1"]
KERNEL_OBJS = ["tcu_tall.o", "tcu_gemm.o", "tcu_poly.o", "tcu_tc.o", "tcu_dft.o"]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"
    return res


def _env(leaks: bool):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = f"detect_leaks={int(leaks)}:verify_asan_link_order=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", "-fopenmp", "-ffp-contract=off", *SAN, "-o", exe,
          os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "tcu_oracle.c"),
          "-lm"])
    res = _run([exe], env=_env(leaks=True))
    assert "0 failures" in res.stdout


@pytest.mark.skipif(shutil.which("g++") is None or torch.cuda.is_available(),
                    reason="needs g++ and a machine without a GPU (valid calls must stop at the "
                           "device query)")
def test_abi_validation_under_asan_ubsan(tmp_path):
    build_dir = os.path.join(ROOT, "_build")
    if not all(os.path.exists(os.path.join(build_dir, o)) for o in KERNEL_OBJS):
        from paper_1908_06649_amd import build as hip_build
        hip_build.build()
    inc = ["-I" + os.path.join(ROOT, "include"),
           "-I" + os.path.join(ROOT, "paper_1908_06649_amd", "csrc")]
    abi_o, drv_o, exe = (str(tmp_path / n) for n in ("abi.o", "drv.o", "abi_driver"))
    _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", *inc, "-c",
          os.path.join(ROOT, "paper_1908_06649_amd", "csrc", "tcu_abi.cpp"), "-o", abi_o])
    _run(["gcc", "-std=c11", *SAN, *inc, "-c", os.path.join(HERE, "abi_driver.c"), "-o", drv_o])
    _run(["g++", *SAN, drv_o, abi_o, *[os.path.join(build_dir, o) for o in KERNEL_OBJS],
          f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", exe])
    res = _run([exe], env=_env(leaks=False))
    assert "0 failures" in res.stdout
