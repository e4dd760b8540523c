"""Compile the HIP library (gfx950) into paper_1908_06649_amd/libtcu.so.

Every source is compiled with hipcc for gfx950 only; packed-fp32 instruction
selection is disabled for all device code.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libtcu.so")
# The benchmark's host-side timing loop (calls libtcu.so through the C ABI).
TIMING_SRC = "tcu_timing.cpp"
TIMING_LIB = os.path.join(HERE, "libtcu_timing.so")
# The benchmark's matrix-core ceiling probe (a kernel of its own, outside the C ABI).
PROBE_SRC = "tcu_probe.hip"
PROBE_LIB = os.path.join(HERE, "libtcu_probe.so")
BUILD_DIR = os.path.join(ROOT, "_build")
SOURCES = ["tcu_abi.cpp", "tcu_tall.hip", "tcu_gemm.hip", "tcu_poly.hip", "tcu_tc.hip",
           "tcu_dft.hip"]
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
          f"--offload-arch={ARCH}", f"-I{INCLUDE}", f"-I{CSRC}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-command-line-argument"]


# Per-source additions.  The polynomial kernel consumes every matrix-core
# result with vector ALU work at once; the VGPR-destination form of the
# instruction saves a register-file move per result value.
EXTRA = {"tcu_poly.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
         "tcu_dft.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def hipcc() -> str:
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *COMMON, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    # host-pass warning about the device-only target feature is expected
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    tmp = TIMING_LIB + ".tmp"
    cmd = [hipcc(), "-O2", "-std=c++17", "-fPIC", "-shared", f"-I{INCLUDE}",
           os.path.join(CSRC, TIMING_SRC), f"-L{HERE}", "-ltcu", "-Wl,-rpath,$ORIGIN",
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {TIMING_SRC}:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, TIMING_LIB)
    tmp = PROBE_LIB + ".tmp"
    cmd = [hipcc(), *COMMON, "-shared", os.path.join(CSRC, PROBE_SRC), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {PROBE_SRC}:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, PROBE_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
