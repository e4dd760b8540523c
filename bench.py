#!/usr/bin/env python3
"""Benchmark of the (m,l)-TCU hot path on one MI355X.

One step is one tcu_gemm call on the headline workload (the blocked product
of Theorem 2, which performs every stage of the path: weights loaded into the
unit, tall strips streamed through it, partial products summed, output
written, calls counted), with inputs already resident in HBM.  Prints ONE
JSON line:

  value      TFLOP/s of tcu_gemm on gemm_bf16_N8192_s32 (A, B 8192 x 8192
             bfloat16 ~ N(0,1), seed 2; unit s = 32; binary32 sums/output)
  roofline   that kernel against the dense bf16 matrix-core peak, with the
             HBM traffic rocprofv3 counted for it (when still current)
  cpu_baseline  the CPU oracle timed on a bounded sample of the same product
             on this host's cores (all rows when they fit ~15 s), and the
             sampled rows' parity; "host" names the CPU model, nproc,
             OMP_NUM_THREADS and the oracle's thread count
  secondary  the other workloads measured the same way: the very tall
             bf16 native call (GB/s vs HBM peak), the int8 product (TOP/s),
             the 4096 x 16 native call and the N = 1024 fp16 product, each
             with its own cpu_baseline (oracle seconds and parity)
  poly       batch polynomial evaluation (tcu_poly_eval, Theorem 11) on 2^24
             points with 4096 coefficients: TFLOP/s of the method's 2pn
             multiply-adds vs the bf16 matrix-core peak
  dft        DFT (tcu_dft, Theorem 7) of 16 complex64 vectors of 2^20: GB/s of
             the launches' traffic (each launch -- one of the ceil(log_32 n)
             levels, or two consecutive levels fused through LDS -- reads and
             writes the array once) vs HBM peak, and 5 n log2 n GFLOP/s
  tc         transitive closure (tcu_transitive_closure, Theorem 5) of a
             random 8192-vertex digraph: GB/s of the D updates' algorithmic
             traffic (each pivot band reads and writes the off-band n^2 bytes)
             vs HBM peak, and boolean TOP/s (2 n^3 / t); every timed call
             starts from the raw graph (restored outside the timed region);
             the oracle's closure timed and compared exactly
  rect       the rectangular / accumulating product (tcu_gemm_rect):
             Corollary 1's sqrt(n) x r by r x sqrt(n) with r below and above
             sqrt(n), accumulating into C, and an order-8200 product that
             needs zero padding (TFLOP/s or TOP/s vs matrix-core peak)
  cost_model calls issued vs Theorem 2's count and bound, weak-model square
             calls, model work; the native call's cost t(n) = a*(n s) + l
             fitted per type pair and unit size from a C timing loop; and per
             configured workload the model time T = a*work + calls*l
             (N^3/s + (N/s)^2 l for the product, n s + l for a native call)
             against the measured time

Timing: every measured call first runs back to back, untimed, for 0.3 s
(the GPU leaves its idle clock state), then W untimed warmup calls, then K
calls bracketed by HIP events on the stream the library launches on.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
       [--no-cpu-baseline] [--no-secondary] [--copy-probe] [--mfma-probe] [--vendor-probe]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("TFLOP/s (or TOP/s) and % MFMA peak for tcu_gemm; "
          "GB/s and % HBM peak for tcu_mm_tall")
HEADLINE = "gemm_bf16_N8192_s32"
# MI355X published peaks (dense): matrix cores by input type, and HBM3E.
PEAK = {"f16": 2500.0, "bf16": 2500.0, "i8": 5000.0}   # TFLOP/s or TOP/s
HBM_PEAK_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_1908_06649_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


def kernel_sources(kind: str):
    main = {"gemm": ["tcu_gemm.hip", "tcu_tc_diag.h"], "rect": ["tcu_gemm.hip", "tcu_tc_diag.h"],
            "poly": ["tcu_poly.hip", "tcu_split.h"],
            "tc": ["tcu_tc.hip", "tcu_gemm.hip", "tcu_tc_diag.h"],
            "dft": ["tcu_dft.hip", "tcu_split.h"],
            "probe": ["tcu_probe.hip"]}.get(kind, ["tcu_tall.hip"])
    return [os.path.join(CSRC, f) for f in (*main, "tcu_device.h")]


def kernel_hash(kind: str) -> str:
    h = hashlib.sha256()
    for p in kernel_sources(kind):
        with open(p, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counted_traffic(name: str, kind: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary of
    this workload, if it was taken on the current kernel source; else None.
    A workload whose call is several launches (the closure) has a summary
    with a per-call total, which is what its per-call rate compares with."""
    path = os.path.join(PROFILES, f"{name}_counters.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as fh:
        for line in fh:
            m = re.match(r"^([a-z_0-9]+):\s*(\S+)", line.strip())
            if m:
                fields[m.group(1)] = m.group(2)
    if fields.get("kernel_source_sha256") != kernel_hash(kind):
        return None
    try:
        return float(fields.get("hbm_bytes_per_call", fields["hbm_bytes_per_dispatch"]))
    except (KeyError, ValueError):
        return None


def dft_levels(n: int, s: int) -> int:
    """Cooley-Tukey levels of radix s (the last of radix <= s) for length n."""
    levels, m = 1, s
    while m < n:
        m *= s
        levels += 1
    return levels


def dft_launches(n: int, s: int) -> int:
    """Launches of tcu_dft for length n with the library's default choice:
    two consecutive full-radix levels in one launch where it pairs them (level
    t+1 of full radix, and P_t >= 16 or P_t = 1 with at least 16 groups per
    vector), else one launch per level.  Each launch reads and writes the
    array once."""
    levels, P, t, launches = dft_levels(n, s), 1, 1, 0
    while t <= levels:
        n2 = n // P // s
        pair = t < levels and n2 >= s and (P >= 16 or (P == 1 and n2 // s >= 16))
        P *= s * s if pair else (s if t < levels else n // P)
        t += 2 if pair else 1
        launches += 1
    return launches


def algorithmic(spec: dict):
    """(work per call in flop/op, bytes per call) that the method must do."""
    ib = 1 if spec.get("dtype", "i8") == "i8" else 2
    ob = 2 if spec.get("out") == "bf16" else 4
    if spec["kind"] == "tall":
        n, s = spec["n"], spec["s"]
        return 2.0 * n * s * s, n * s * ib + s * s * ib + n * s * ob
    if spec["kind"] == "dft":
        n, b = spec["n"], spec["batch"]
        return 5.0 * b * n * math.log2(n), dft_launches(n, spec["s"]) * 2 * 8 * b * n
    if spec["kind"] == "tc":
        # per pivot band of up to 256 vertices: the D update reads and writes
        # every off-band entry once, the panel updates their band entries
        n = spec["n"]
        nbytes = 0
        for k0 in range(0, n, 256):
            bk = min(256, n - k0)
            nbytes += 2 * (n - bk) ** 2 + 2 * 2 * bk * (n - bk) + 2 * bk * bk
        return 2.0 * n ** 3, nbytes + 2 * n * n          # + the normalizing pass
    if spec["kind"] == "poly":
        n, p = spec["n"], spec["p"]
        return 2.0 * n * p, n * ib + p * ib + p * ob
    if spec["kind"] == "rect":
        M, K, N = spec["M"], spec["K"], spec["N"]
        c_io = 2 if spec.get("acc") else 1          # C read too when accumulating
        return 2.0 * M * K * N, (M * K + K * N) * ib + c_io * M * N * ob
    N = spec["N"]
    return 2.0 * N ** 3, 2 * N * N * ib + N * N * ob


class Workload:
    """Inputs of one workload resident on the device, plus the call."""

    def __init__(self, name: str):
        import torch
        from paper_1908_06649_amd import inputs, tcu
        self.name = name
        self.spec = (inputs.WORKLOADS.get(name) or inputs.RECT_WORKLOADS.get(name)
                     or inputs.POLY_WORKLOADS.get(name) or inputs.TC_WORKLOADS.get(name)
                     or inputs.DFT_WORKLOADS[name])
        self.tcu = tcu
        self.s = self.spec["s"]
        if self.spec["kind"] == "dft":
            sp = self.spec
            self.A = inputs.complex_signal(sp["batch"], sp["n"], sp["seed"])
            self.dA = self.A.cuda()
            self.C = torch.empty_like(self.dA)
            self.W = torch.empty_like(self.dA)
            return
        if self.spec["kind"] == "tc":
            # The closure is computed in place, and its 0/1 epilogues skip the
            # chunks whose OR changes nothing, so a call on an already closed
            # matrix does less work: every timed call starts from the raw
            # graph, restored from a pristine device copy outside the timing.
            self.A = inputs.make_tc_input(self.spec)
            self.dA = self.A.cuda()
            self.raw = self.dA.clone()
            return
        if self.spec["kind"] == "poly":
            self.A, self.B = inputs.make_poly_inputs(self.spec)     # coefficients, points
            self.dA, self.dB = self.A.cuda(), self.B.cuda()
            self.C = torch.empty(self.spec["p"], dtype=inputs.TORCH_DTYPE[self.spec["out"]],
                                 device="cuda")
            return
        self.A, self.B = inputs.make_inputs(self.spec)
        self.dA, self.dB = self.A.cuda(), self.B.cuda()
        _, _, c_shape = inputs.shapes(self.spec)
        if self.spec.get("acc"):
            self.C = inputs.make_c0(self.spec).cuda()
        else:
            self.C = torch.empty(c_shape, dtype=inputs.TORCH_DTYPE[self.spec["out"]],
                                 device="cuda")
        self.s = self.spec["s"]

    def restore(self):
        """Put the raw input back (the in-place closure only; else None)."""
        self.dA.copy_(self.raw)

    def needs_restore(self) -> bool:
        return self.spec["kind"] == "tc"

    def call(self):
        sp = self.spec
        if sp["kind"] == "gemm":
            self.tcu.tcu_gemm(self.dA, self.dB, self.C, sp["N"])
        elif sp["kind"] == "dft":
            self.tcu.tcu_dft(self.dA, self.C, self.W, sp["n"], sp["batch"])
        elif sp["kind"] == "tc":
            self.tcu.tcu_transitive_closure(self.dA, sp["n"], sp["n"])
        elif sp["kind"] == "poly":
            self.tcu.tcu_poly_eval(self.dA, sp["n"], self.dB, sp["p"], self.C)
        elif sp["kind"] == "rect":
            M, K, N = sp["M"], sp["K"], sp["N"]
            self.tcu.tcu_gemm_rect(self.dA, K, self.dB, N, self.C, N, M, K, N,
                                   self.tcu.TCU_ACCUMULATE if sp["acc"] else 0)
        else:
            self.tcu.tcu_mm_tall(self.dA, sp["n"], sp["s"], self.dB, self.C)


SETTLE_S = 0.3


def settle(fn, seconds: float = SETTLE_S, restore=None) -> None:
    """Run the call back to back for `seconds` (untimed) so the GPU leaves
    its idle clock state: after the host-side input generation the device has
    been idle, and the first milliseconds of work run measurably slower."""
    import torch
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            if restore is not None:
                restore()
            fn()
        torch.cuda.synchronize()


def time_steps(fn, steps: int, warmup: int, restore=None) -> float:
    """Average ms per call over `steps` calls, timed with HIP events on the
    current stream (the stream the library launches on), after a
    clock-settling period and `warmup` untimed calls.  Without `restore` the
    calls run back to back between one pair of events; with it, every call
    is preceded by restore() (putting an in-place call's input back) outside
    its own pair of events, and the per-call times are summed."""
    import torch
    settle(fn, restore=restore)
    for _ in range(warmup):
        if restore is not None:
            restore()
        fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    if restore is None:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(steps):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps
    pairs = []
    for _ in range(steps):
        restore()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        fn()
        e1.record(st)
        pairs.append((e0, e1))
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in pairs) / steps


def measure(name: str, steps: int, warmup: int) -> dict:
    w = Workload(name)
    tcu = w.tcu
    tcu.tcu_set_unit(w.s)
    restore = w.restore if w.needs_restore() else None
    ms = time_steps(w.call, steps, warmup, restore=restore)
    tcu.tcu_reset_calls()
    if restore is not None:
        restore()
    w.call()
    import torch
    torch.cuda.synchronize()
    calls, squares, work = tcu.tcu_calls(), tcu.tcu_square_calls(), tcu.tcu_work()
    flops, nbytes = algorithmic(w.spec)
    sp = w.spec
    kind = sp["kind"]
    out = {"workload": name, "ms_per_call": ms, "calls": calls, "square_calls": squares,
           "model_work": work}
    if kind == "dft":
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.update({"value": gbs, "unit": "GB/s",
                    "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS,
                                 "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                                 "traffic": counted_traffic(name, kind)},
                    "gflops_5nlogn": flops / (ms * 1e-3) / 1e9,
                    "levels": dft_levels(sp["n"], sp["s"]),
                    "launches_per_call": dft_launches(sp["n"], sp["s"]),
                    "algorithmic_bytes_per_launch": nbytes / dft_launches(sp["n"], sp["s"])})
    elif kind == "tc":
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.update({"value": gbs, "unit": "GB/s",
                    "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS,
                                 "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                                 "traffic": counted_traffic(name, kind)},
                    "bool_tops": flops / (ms * 1e-3) / 1e12,
                    "algorithmic_bytes": nbytes,
                    "calls_section43": (-(-sp["n"] // sp["s"])) * (-(-sp["n"] // sp["s"]) - 1)})
    elif kind in ("gemm", "rect", "poly"):
        tput = flops / (ms * 1e-3) / 1e12
        peak = PEAK[sp["dtype"]]
        out.update({"value": tput, "unit": "TOP/s" if sp["dtype"] == "i8" else "TFLOP/s",
                    "roofline": {"bound": "mfma", "achieved": tput, "peak": peak,
                                 "unit": "TOP/s" if sp["dtype"] == "i8" else "TFLOP/s",
                                 "frac": tput / peak,
                                 "traffic": counted_traffic(name, kind)},
                    "algorithmic_flops": flops, "compulsory_bytes": nbytes})
        if kind == "gemm":
            out["calls_theorem2"] = (sp["N"] // sp["s"]) ** 2
        elif kind == "poly":   # Theorem 11's n/m calls, each issued for X_hi and X_lo
            out["calls_theorem11"] = 2 * -(-sp["n"] // (sp["s"] * sp["s"]))
            out["points_per_s"] = sp["p"] / (ms * 1e-3)
        else:   # Corollary 1 on the zero-padded operands
            out["calls_corollary1"] = -(-sp["K"] // sp["s"]) * -(-sp["N"] // sp["s"])
    else:
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.update({"value": gbs, "unit": "GB/s",
                    "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS,
                                 "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                                 "traffic": counted_traffic(name, kind)},
                    "tflops": flops / (ms * 1e-3) / 1e12,
                    "algorithmic_bytes": nbytes, "algorithmic_flops": flops})
    out["_workload"] = w
    return out


# (dtype code, unit size) of the native calls whose cost is fitted, keyed by
# the (input, output) types of the configured workloads.
ELL_CASES = {("f16", "f32"): 16, ("bf16", "f32"): 32, ("bf16", "bf16"): 32, ("i8", "i32"): 32}
ELL_ROWS = [16, 32, 256, 1024, 4096, 16384, 65536, 262144, 1048576, 4194304, 16777216]


def _timing_lib():
    import ctypes
    from paper_1908_06649_amd import build as hip_build
    if not os.path.exists(hip_build.TIMING_LIB):
        raise RuntimeError(f"{hip_build.TIMING_LIB} is missing: build the library first")
    lib = ctypes.CDLL(hip_build.TIMING_LIB)
    fn = lib.tcu_timing_tall_loop
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                   ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                   ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    return fn


def ell_fit() -> dict:
    """The model's cost of one native call, O(n sqrt(m) + l) (Section 3),
    fitted per (input, output) type and unit size as t(n) = a*(n*s) + l: a
    in seconds per unit of model work, l the per-call latency.  Times come
    from a loop in C (libtcu_timing.so) issuing tcu_mm_tall_ex back to back
    on torch's current stream, so no Python marshalling is in them; the fit
    weights each point by 1/t (relative residuals), so the small-n points fix
    l and the large-n points fix a.  Also reported: the round trip of one
    synchronised call, and the Python binding's per-call time at the
    smallest n for comparison."""
    import ctypes
    import numpy as np
    import torch
    from paper_1908_06649_amd import inputs, tcu
    loop = _timing_lib()
    st = torch.cuda.current_stream().cuda_stream
    codes = {("f16", "f32"): tcu.TCU_F16_F32, ("bf16", "f32"): tcu.TCU_BF16_F32,
             ("bf16", "bf16"): tcu.TCU_BF16_BF16, ("i8", "i32"): tcu.TCU_I8_I32}
    out = {}
    for (din, dout), s in ELL_CASES.items():
        ns = [n for n in ELL_ROWS if n >= s]
        nmax = ns[-1]
        g = torch.Generator().manual_seed(99)
        A = inputs.draw((nmax, s), din, "int8" if din == "i8" else "normal", g).cuda()
        B = inputs.draw((s, s), din, "int8" if din == "i8" else "normal", g).cuda()
        C = torch.empty(nmax, s, dtype=inputs.TORCH_DTYPE[dout], device="cuda")
        ts, tsync = [], []
        settle(lambda: tcu.tcu_mm_tall_ex(A, nmax, s, B, C), 0.2)
        for n in ns:
            reps = max(20, min(2000, int(2e7 // (n * s))))
            a_t, s_t = ctypes.c_double(), ctypes.c_double()
            rc = loop(A.data_ptr(), n, s, B.data_ptr(), C.data_ptr(), codes[(din, dout)], st,
                      reps, ctypes.byref(a_t), ctypes.byref(s_t))
            if rc != 0:
                raise RuntimeError(f"timing loop failed: {tcu.tcu_strerror(rc)}")
            ts.append(a_t.value)
            tsync.append(s_t.value)
        x = np.array(ns, dtype=float) * s
        y = np.array(ts)
        w = 1.0 / y
        slope, icpt = np.polyfit(x, y, 1, w=w)
        n0 = ns[0]
        a0, c0 = A[:n0], C[:n0]
        py_ms = time_steps(lambda: tcu.tcu_mm_tall_ex(a0, n0, s, B, c0), 500, 20)
        out[f"{din}_{dout}_s{s}"] = {
            "s": s, "n": ns, "us_per_call_async": [round(t * 1e6, 3) for t in ts],
            "us_per_call_sync": [round(t * 1e6, 3) for t in tsync],
            "a_s_per_work": float(slope), "ell_us": float(icpt) * 1e6,
            "python_binding_us_per_call_at_min_n": py_ms * 1e3}
        del A, B, C
        torch.cuda.empty_cache()
    return out


def model_time(spec: dict, calls: int, work: int, ms: float, fits: dict) -> dict | None:
    """Theorem 2's (and the native call's) model time for one call of the
    workload -- T = a * (model work) + (calls) * l, with a and l fitted for
    its types and unit size (ell_fit) -- against the measured time."""
    key = f"{spec.get('dtype')}_{spec.get('out')}_s{spec.get('s')}"
    f = fits.get(key)
    if f is None:
        return None
    t_model = f["a_s_per_work"] * work + calls * f["ell_us"] * 1e-6
    form = ("N^3/s + (N/s)^2 l" if spec["kind"] == "gemm" else
            "n s + l" if spec["kind"] == "tall" else "work + calls l")
    return {"form": form, "fit": key, "model_work": work, "calls": calls,
            "a_s_per_work": f["a_s_per_work"], "ell_us": f["ell_us"],
            "T_model_ms": t_model * 1e3, "measured_ms": ms,
            "measured_over_model": (ms * 1e-3) / t_model if t_model > 0 else None}


def host_info() -> dict:
    """The machine the CPU oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = None
    import oracle
    return {"cpu_model": model, "nproc": os.cpu_count(), "affinity_cpus": affinity,
            "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS"),
            "oracle_threads": oracle.threads()}


def cpu_baseline(w: "Workload", target_s: float = 15.0) -> dict | None:
    """Time the CPU oracle on a bounded sample of the workload just measured
    and compare the GPU result with it on that sample.
      product / native call: R of the output rows (R rows of A times B), R
        sized from two probes for ~target_s seconds (all rows when they fit);
      closure: the whole closure (bit sets, the section's iterative
        algorithm), compared exactly.
    Parity on the sample: bit-exact for int8, else the relative Frobenius,
    elementwise and (bfloat16 output) rounding bounds of oracle/compare."""
    import numpy as np
    import oracle
    from oracle import compare
    from paper_1908_06649_amd import inputs
    sp = w.spec
    if sp["kind"] == "tc":
        d = w.A.numpy()
        t0 = time.perf_counter()
        ref = oracle.transitive_closure(d)
        secs = time.perf_counter() - t0
        got = w.dA.cpu().numpy().view(np.uint8)
        mism = int((got != ref).sum())
        assert mism == 0, f"closure differs from the oracle in {mism} entries"
        n = sp["n"]
        return {"value": 2.0 * n ** 3 / secs / 1e12, "unit": "boolean TOP/s",
                "cores": oracle.threads(), "kind": "oracle",
                "sample": f"the whole closure of the {n}-vertex graph, bit-set rows",
                "seconds": secs, "parity": {"mismatches": 0}}
    if sp["kind"] not in ("gemm", "tall"):
        return None
    dt, out = sp["dtype"], sp["out"]
    Ab, Bb = inputs.bits(w.A), inputs.bits(w.B)
    rows_total, K = Ab.shape
    J = Bb.shape[1]
    rng = np.random.default_rng(123)
    # two probes separate the per-call setup (decoding B) from the per-row cost
    t_probe = []
    for k in (8, 40):
        k = min(k, rows_total)
        rows_p = np.sort(rng.choice(rows_total, k, replace=False))
        t0 = time.perf_counter()
        oracle.mm(Ab, Bb, dt, rows=rows_p)
        t_probe.append(time.perf_counter() - t0)
    per_row = max((t_probe[1] - t_probe[0]) / 32, 1e-9)
    fixed = max(t_probe[0] - 8 * per_row, 0.0)
    R = int(max(8, min(rows_total, (target_s - fixed) / per_row)))
    rows = None if R >= rows_total else np.sort(rng.choice(rows_total, R, replace=False))
    R = rows_total if rows is None else R
    t0 = time.perf_counter()
    ref = oracle.mm(Ab, Bb, dt, rows=rows)
    secs = time.perf_counter() - t0
    Cg = w.C.view(rows_total, J)
    got = Cg if rows is None else Cg[rows]
    got = got.cpu()
    got = got.view(__import__("torch").int16).numpy().view(np.uint16) if out == "bf16" \
        else got.numpy()
    if dt == "i8":
        parity = compare.check_exact(got, ref)
    else:
        absab = oracle.mm(compare.abs_bits(Ab), compare.abs_bits(Bb), dt, rows=rows)
        parity = (compare.check_bf16(got, ref, absab, K=K) if out == "bf16"
                  else compare.check_float(got, ref, absab))
    flops = 2.0 * R * K * J
    what = (f"{sp['N']}x{sp['N']} {dt} product" if sp["kind"] == "gemm"
            else f"{rows_total}x{K} by {K}x{J} {dt} native call")
    return {"value": flops / secs / 1e12, "unit": "TOP/s" if dt == "i8" else "TFLOP/s",
            "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{R} of {rows_total} output rows of the {what} ({flops:.3e} "
                      f"{'op' if dt == 'i8' else 'flop'}), binary64/int64 triple loop",
            "seconds": secs, "parity_sampled_rows": parity}


def copy_probe() -> None:
    """A plain device copy of known size (1 GiB), for calibrating rocprofv3's
    FETCH_SIZE / WRITE_SIZE counters (the first 3 copies), then timed (20
    more, after a settle) as the rate a plain stream reaches on this GPU:
    the practical ceiling of the HBM-bound kernels."""
    import torch
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    ms = time_steps(lambda: dst.copy_(src), 20, 3)
    print(json.dumps({"copy_probe_bytes_each_way": nbytes, "copies": 3,
                      "timed_copies": 20, "ms_per_copy": ms,
                      "GB_per_s_read_plus_write": 2 * nbytes / (ms * 1e-3) / 1e9}))


def vendor_probe(steps: int = 50, warmup: int = 5, passes: int = 2) -> None:
    """Reference rates of the vendor BLAS on this GPU (hipBLASLt, reached
    through torch.mm with out_dtype=float32 and torch._int_mm) for the square
    products gemm_bf16_N8192_s32 (bfloat16 in, binary32 out) and
    gemm_i8_N8192_s32 (int8 in, int32 out): the same device-resident inputs,
    timed the same way and alternated with this library's tcu_gemm in one
    process.  Context for the products' rates only -- nothing of the library
    calls it.  Prints one JSON line."""
    import torch
    res = {"probe": "vendor BLAS reference (torch.mm / torch._int_mm -> hipBLASLt)",
           "steps": steps, "warmup": warmup, "passes": []}
    for _ in range(passes):
        one = {}
        for name in ("gemm_bf16_N8192_s32", "gemm_i8_N8192_s32"):
            w = Workload(name)
            w.tcu.tcu_set_unit(w.s)
            N = w.spec["N"]
            ours = time_steps(w.call, steps, warmup)
            if w.spec["dtype"] == "bf16":
                cv = torch.empty(N, N, dtype=torch.float32, device="cuda")
                vendor_call = lambda: torch.mm(w.dA, w.dB, out_dtype=torch.float32, out=cv)  # noqa: E731
            else:
                holder = {}
                vendor_call = lambda: holder.__setitem__("c", torch._int_mm(w.dA, w.dB))  # noqa: E731
            vendor = time_steps(vendor_call, steps, warmup)
            w.call()
            vendor_call()
            torch.cuda.synchronize()
            ref = cv if w.spec["dtype"] == "bf16" else holder["c"]
            diff = (w.C.double() - ref.double()).abs().max().item()
            scale = ref.double().abs().max().item()
            flops = 2.0 * N ** 3
            one[name] = {"tcu_gemm_ms": ours, "vendor_ms": vendor,
                         "tcu_gemm_T_per_s": flops / (ours * 1e-3) / 1e12,
                         "vendor_T_per_s": flops / (vendor * 1e-3) / 1e12,
                         "max_abs_difference": diff, "max_abs_value": scale}
            del w
        res["passes"].append(one)
    print(json.dumps(res), flush=True)


def mfma_probe(iters: int = 100000, reps: int = 3) -> None:
    """The matrix cores' sustained rate on this chip with nothing else
    running (libtcu_probe.so: the product's persistent grid, one workgroup of
    8 waves per CU, each wave issuing the product's 32-instruction phase from
    registers `iters` times), for bfloat16 and int8 operands drawn at random
    as in the workloads and for constant operands: the power-limited ceiling
    the products are measured against.  Prints one JSON line."""
    import ctypes
    import torch
    from paper_1908_06649_amd import build as hip_build
    from paper_1908_06649_amd import tcu
    lib = ctypes.CDLL(hip_build.PROBE_LIB)
    fn = lib.tcu_probe_mfma
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                   ctypes.c_void_p]
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    words = blocks * 512 * 12 * 4                 # 12 16-byte operands per lane
    g = torch.Generator(device="cuda").manual_seed(77)
    out = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
    res = {"probe": "matrix-core ceiling", "blocks": blocks, "waves_per_block": 8,
           "instructions_per_wave": 32 * iters}
    st = torch.cuda.current_stream()
    for name, dt, peak in (("bf16", tcu.TCU_BF16_F32, PEAK["bf16"]),
                           ("i8", tcu.TCU_I8_I32, PEAK["i8"])):
        for kind in ("random", "constant"):
            if kind == "constant":
                ops = torch.full((words,), 0x3F803F80 if name == "bf16" else 0x01010101,
                                 dtype=torch.int32, device="cuda")
            elif name == "bf16":
                ops = torch.randn(words * 2, generator=g, device="cuda").to(torch.bfloat16)
                ops = ops.view(torch.int32)
            else:
                ops = torch.randint(-128, 128, (words * 4,), generator=g, device="cuda",
                                    dtype=torch.int8).view(torch.int32)
            assert ops.numel() == words and out.numel() == blocks * 512

            def run():
                rc = fn(dt, ops.data_ptr(), out.data_ptr(), iters, blocks, st.cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"probe launch failed ({rc})")

            run()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            for _ in range(reps):
                run()
            e1.record(st)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            flops = blocks * 8 * 32 * iters * (16 * 16 * 32 * 2 if name == "bf16" else
                                               16 * 16 * 64 * 2)
            rate = flops / (ms * 1e-3) / 1e12
            res[f"{name}_{kind}"] = {"ms": ms, "T_per_s": rate, "frac_of_peak": rate / peak}
    res["overlap"] = overlap_probe(lib, blocks, st)
    res["lds"] = lds_probe(lib, blocks, st)
    res["dma"] = dma_probe(lib, blocks, st)
    res["pingpong"] = pingpong_probe(lib, blocks, st)
    print(json.dumps(res), flush=True)


def _timed_launch(run, st, reps: int) -> float:
    """Milliseconds per launch: one untimed launch, then `reps` between events."""
    import torch
    run()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(reps):
        run()
    e1.record(st)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def dma_probe(lib, blocks: int, st, iters: int = 20000, reps: int = 3) -> dict:
    """Rate of direct global -> LDS loads per CU (libtcu_probe.so,
    tcu_probe_dma; one workgroup of 4, 8 or 16 waves per CU, each wave 4
    loads of 1 KiB per round from a cache-resident window), in bytes per ns
    per CU."""
    import ctypes
    import torch
    fn = lib.tcu_probe_dma
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                   ctypes.c_void_p]
    src = torch.ones(1 << 18, dtype=torch.int32, device="cuda")      # 1 MiB (>= 512 KiB read)
    out = torch.empty(blocks * 1024, dtype=torch.int32, device="cuda")
    res = {"iters": iters}
    for threads in (256, 512, 1024):
        def run():
            rc = fn(src.data_ptr(), out.data_ptr(), iters, blocks, threads, st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"dma probe launch failed ({rc})")
        ms = _timed_launch(run, st, reps)
        nbytes = (threads // 64) * iters * 4 * 1024          # per CU
        res[f"waves{threads // 64}"] = {"ms": ms, "bytes_per_ns_per_cu": nbytes / (ms * 1e6)}
    return res


def pingpong_probe(lib, blocks: int, st, iters: int = 20000, reps: int = 3) -> dict:
    """The full-tile product's two-group phase structure with its parts added
    one at a time (libtcu_probe.so, tcu_probe_pingpong; one workgroup of 8
    waves per CU, products from registers): nanoseconds per matrix-core
    instruction per SIMD for no ping-pong, ping-pong with barriers only, +
    the other group's fragment reads, + its DMA loads (the product's phase),
    and the DMA loads without the reads."""
    import ctypes
    import torch
    fn = lib.tcu_probe_pingpong
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int, ctypes.c_void_p]
    g = torch.Generator(device="cuda").manual_seed(79)
    ops = torch.randn(blocks * 2048 * 8, generator=g, device="cuda").to(torch.bfloat16)
    ops = ops.view(torch.int32)
    assert ops.numel() == blocks * 2048 * 4
    src = torch.zeros(1 << 18, dtype=torch.int32, device="cuda")     # 1 MiB
    out = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
    res = {"iters": iters}
    names = ("no_pingpong", "pingpong_barriers", "plus_fragment_reads", "plus_dma_product_phase",
             "dma_without_reads")
    for mode, name in enumerate(names):
        def run():
            rc = fn(mode, ops.data_ptr(), src.data_ptr(), out.data_ptr(), iters, blocks,
                    st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"pingpong probe launch failed ({rc})")
        ms = _timed_launch(run, st, reps)
        res[name] = {"ms": ms, "ns_per_product_per_simd": ms * 1e6 / (64 * iters)}
    return res


def lds_probe(lib, blocks: int, st, iters: int = 20000, reps: int = 3) -> dict:
    """LDS read rate per CU (libtcu_probe.so, tcu_probe_lds; one workgroup of
    4, 8 or 16 waves per CU, 16 reads per wave and round): ds_read_b128 (1 KiB
    per instruction), ds_read_b64_tr_b16 and ds_read_b64_tr_b8 (512 bytes;
    the 16-bit and int8 products' weights reads), in bytes per ns per CU and
    ns per instruction per CU."""
    import ctypes
    import torch
    fn = lib.tcu_probe_lds
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                   ctypes.c_void_p]
    out = torch.empty(blocks * 1024, dtype=torch.int32, device="cuda")
    res = {"iters": iters}
    for kind, name, nbytes in ((0, "b128", 1024), (1, "tr16_b64", 512), (2, "tr8_b64", 512)):
        for threads in (256, 512, 1024):
            def run():
                rc = fn(kind, out.data_ptr(), iters, blocks, threads, st.cuda_stream)
                if rc != 0:
                    raise RuntimeError(f"lds probe launch failed ({rc})")
            run()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            for _ in range(reps):
                run()
            e1.record(st)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            instr = (threads // 64) * iters * 16        # per CU
            res[f"{name}_waves{threads // 64}"] = {
                "ms": ms, "bytes_per_ns_per_cu": instr * nbytes / (ms * 1e6),
                "ns_per_instruction_per_cu": ms * 1e6 / instr}
    return res


def overlap_probe(lib, blocks: int, st, iters: int = 10000, reps: int = 3) -> dict:
    """Whether binary32 vector FMAs run while the matrix core works
    (libtcu_probe.so, tcu_probe_overlap; one workgroup of 8 waves per CU):
    `same_wave` -- every wave issues 32 bfloat16 matrix-core instructions
    per round, each followed by nv independent FMAs; `mfma_waves` /
    `valu_waves` / `both` -- waves 0-3 issue only the 32 matrix-core
    instructions per round, waves 4-7 (on the same SIMDs) only 32 nv FMAs,
    each kind alone and both at once.  Milliseconds per launch of `iters`
    rounds."""
    import ctypes
    import torch
    fn = lib.tcu_probe_overlap
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int, ctypes.c_void_p]
    g = torch.Generator(device="cuda").manual_seed(78)
    ops = torch.randn(blocks * 512 * 3 * 8, generator=g, device="cuda").to(torch.bfloat16)
    ops = ops.view(torch.int32)
    out = torch.empty(blocks * 512, dtype=torch.int32, device="cuda")
    assert ops.numel() == blocks * 512 * 3 * 4

    def timed(mode, nv):
        def run():
            rc = fn(mode, nv, ops.data_ptr(), out.data_ptr(), iters, blocks, st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"overlap probe launch failed ({rc})")
        run()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            run()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    res = {"iters": iters, "same_wave": {}, "separate_waves": {}}
    for nv in (0, 1, 2, 3, 4, 6):
        res["same_wave"][f"nv{nv}"] = timed(0, nv)
    for nv in (2, 4, 6):
        res["separate_waves"][f"nv{nv}"] = {"mfma_waves": timed(2, nv), "valu_waves": timed(3, nv),
                                            "both": timed(1, nv)}
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--no-rect", action="store_true")
    ap.add_argument("--no-poly", action="store_true")
    ap.add_argument("--no-tc", action="store_true")
    ap.add_argument("--no-dft", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--mfma-probe", action="store_true")
    ap.add_argument("--vendor-probe", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the library "
              "has no multi-GPU path (its calls need no collectives; rows shard with no "
              "exchange).", file=sys.stderr)
        return 2
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no HIP device visible", file=sys.stderr)
        return 2
    from paper_1908_06649_amd import inputs, tcu
    tcu.lib()   # raises if the HIP library is missing: no fallback
    if args.copy_probe:
        copy_probe()
        return 0
    if args.mfma_probe:
        mfma_probe()
        return 0
    if args.vendor_probe:
        vendor_probe()
        return 0
    known = {**inputs.WORKLOADS, **inputs.RECT_WORKLOADS, **inputs.POLY_WORKLOADS,
             **inputs.TC_WORKLOADS, **inputs.DFT_WORKLOADS}
    if args.workload not in known:
        names = sorted(known)
        print(f"unknown workload {args.workload}; choose from {names}", file=sys.stderr)
        return 2

    main_res = measure(args.workload, args.steps, args.warmup)
    w = main_res.pop("_workload")
    sp = w.spec
    result = {
        "metric": METRIC,
        "value": main_res["value"],
        "unit": main_res["unit"],
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_call"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": sp.get("dtype", "c64" if sp["kind"] == "dft" else "u8"),
        "data": "synthetic (seeded i.i.d. matrices; the paper has no datasets)",
        "config": {"workload": args.workload,
                   **{k: sp[k] for k in ("kind", "M", "K", "N", "n", "p", "s", "acc", "deg")
                      if k in sp},
                   "dtype_in": sp.get("dtype", "u8"), "dtype_out": sp.get("out", "u8"),
                   "distribution": sp.get("dist", {"poly": "coefficients N(0,1), points U[-1,1)",
                                                   "tc": "random digraph",
                                                   "dft": "re, im ~ N(0,1)"}.get(sp["kind"])),
                   "seed": sp["seed"]},
        "roofline": main_res["roofline"],
    }
    cost = {k: main_res[k] for k in ("calls", "square_calls", "model_work") if k in main_res}
    if sp["kind"] == "gemm":
        cost["calls_theorem2_and_lower_bound"] = main_res["calls_theorem2"]
    elif sp["kind"] == "rect":
        cost["calls_corollary1"] = main_res["calls_corollary1"]
    if not args.no_cpu_baseline and sp["kind"] in ("gemm", "tall", "tc"):
        result["cpu_baseline"] = cpu_baseline(w)
        result["host"] = host_info()
    else:
        result["cpu_baseline"] = None
    del w
    torch.cuda.empty_cache()

    fits = ell_fit() if not args.no_secondary else {}
    if fits:
        cost["ell_fit"] = fits
        mt = model_time(sp, main_res["calls"], main_res["model_work"], main_res["ms_per_call"],
                        fits)
        if mt is not None:
            cost["model_time"] = {args.workload: mt}
    if not args.no_secondary:
        sec = {}
        for name in inputs.WORKLOADS:
            if name == args.workload:
                continue
            spec = inputs.WORKLOADS[name]
            steps = args.steps if spec.get("N", 0) >= 8192 or spec.get("n", 0) >= 1 << 20 else 200
            r = measure(name, steps, max(args.warmup, 5))
            rw = r.pop("_workload")
            sec[name] = {k: r[k] for k in ("value", "unit", "ms_per_call", "roofline", "calls",
                                           "square_calls", "model_work")}
            mt = model_time(spec, r["calls"], r["model_work"], r["ms_per_call"], fits)
            if mt is not None:
                cost.setdefault("model_time", {})[name] = mt
            if not args.no_cpu_baseline:
                sec[name]["cpu_baseline"] = cpu_baseline(rw)
            del rw
            torch.cuda.empty_cache()
        result["secondary"] = sec
    if not args.no_rect:
        rect = {}
        for name in inputs.RECT_WORKLOADS:
            if name == args.workload:
                continue
            r = measure(name, args.steps, max(args.warmup, 5))
            r.pop("_workload")
            rect[name] = {k: r[k] for k in ("value", "unit", "ms_per_call", "roofline", "calls",
                                            "calls_corollary1", "square_calls", "model_work")}
            torch.cuda.empty_cache()
        result["rect"] = rect
    if not args.no_poly:
        poly = {}
        for name in inputs.POLY_WORKLOADS:
            if name == args.workload:
                continue
            r = measure(name, args.steps, max(args.warmup, 5))
            r.pop("_workload")
            poly[name] = {k: r[k] for k in ("value", "unit", "ms_per_call", "roofline", "calls",
                                            "calls_theorem11", "points_per_s", "square_calls",
                                            "model_work")}
            torch.cuda.empty_cache()
        result["poly"] = poly
    if not args.no_tc:
        tc = {}
        for name in inputs.TC_WORKLOADS:
            if name == args.workload:
                continue
            r = measure(name, args.steps, max(args.warmup, 5))
            rw = r.pop("_workload")
            tc[name] = {k: r[k] for k in ("value", "unit", "ms_per_call", "roofline", "bool_tops",
                                          "calls", "calls_section43", "square_calls",
                                          "model_work")}
            tc[name]["timing"] = "each timed call starts from the raw graph (restored outside " \
                                 "the timed region)"
            if not args.no_cpu_baseline:
                tc[name]["cpu_baseline"] = cpu_baseline(rw)
            del rw
            torch.cuda.empty_cache()
        result["tc"] = tc
    if not args.no_dft:
        dft = {}
        for name in inputs.DFT_WORKLOADS:
            if name == args.workload:
                continue
            r = measure(name, args.steps, max(args.warmup, 5))
            r.pop("_workload")
            dft[name] = {k: r[k] for k in ("value", "unit", "ms_per_call", "roofline",
                                           "gflops_5nlogn", "launches_per_call",
                                           "algorithmic_bytes_per_launch", "calls",
                                           "square_calls", "model_work")}
            torch.cuda.empty_cache()
        result["dft"] = dft
    result["cost_model"] = cost
    result["kernel_source_sha256"] = {"gemm": kernel_hash("gemm"), "tall": kernel_hash("tall"),
                                      "poly": kernel_hash("poly"), "tc": kernel_hash("tc"),
                                      "dft": kernel_hash("dft")}
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
