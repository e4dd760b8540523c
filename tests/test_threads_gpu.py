"""Concurrent host threads on the stateful C ABI: each thread sets its own
unit size, dtype and stream (the configuration is per thread) and issues
native calls and blocked products on its own torch stream while the others
do the same; every result must match the oracle, and the call counter
(shared, atomic) must count every call exactly once."""
import threading

import numpy as np
import pytest
import torch

from oracle import compare
from paper_1908_06649_amd import inputs, tcu

import gpu_util as gu

pytestmark = pytest.mark.gpu

# (input, output, unit size, product order, tall rows) per thread
JOBS = [("f16", "f32", 16, 256, 1000), ("bf16", "f32", 32, 512, 777),
        ("bf16", "bf16", 32, 256, 4099), ("i8", "i32", 16, 320, 2048),
        ("i8", "i32", 32, 384, 65)]
ROUNDS = 6


def test_threads_with_their_own_unit_dtype_and_stream():
    dev = torch.device(gu.DEV, torch.cuda.current_device())
    work = []
    for t, (din, dout, s, N, n) in enumerate(JOBS):
        dist = "int8" if din == "i8" else "normal"
        g = torch.Generator().manual_seed(100 + t)
        A = inputs.draw((N, N), din, dist, g)
        B = inputs.draw((N, N), din, dist, g)
        T = inputs.draw((n, s), din, dist, g)
        W = inputs.draw((s, s), din, dist, g)
        work.append(dict(din=din, dout=dout, s=s, N=N, n=n, A=A, B=B, T=T, W=W))
    torch.cuda.synchronize()
    tcu.tcu_reset_calls()
    errors = []
    barrier = threading.Barrier(len(JOBS))

    def run(job):
        try:
            torch.cuda.set_device(dev)
            st = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(st):
                dA, dB = job["A"].to(dev), job["B"].to(dev)
                dT, dW = job["T"].to(dev), job["W"].to(dev)
                od = gu.out_dtype(job["dout"])
                C = torch.empty((job["N"], job["N"]), dtype=od, device=dev)
                Ct = torch.empty((job["n"], job["s"]), dtype=od, device=dev)
                barrier.wait()
                for _ in range(ROUNDS):
                    tcu.tcu_set_unit(job["s"])           # this thread's unit size
                    tcu.tcu_gemm(dA, dB, C, job["N"])
                    tcu.tcu_mm_tall(dT, job["n"], job["s"], dW, Ct)
                    assert tcu.tcu_get_unit() == job["s"]
                st.synchronize()
                job["C"], job["Ct"] = gu.to_np(C), gu.to_np(Ct)
        except Exception as e:          # reported from the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(job,)) for job in work]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not any(th.is_alive() for th in threads), "a thread did not finish"
    assert not errors, errors
    for job in work:
        rows = np.arange(0, job["N"], 7)
        compare.check(job["din"], job["dout"], inputs.bits(job["A"]), inputs.bits(job["B"]),
                      job["C"][rows], rows=rows)
        compare.check(job["din"], job["dout"], inputs.bits(job["T"]), inputs.bits(job["W"]),
                      job["Ct"])
    # every call counted once: a product of order N with unit s is (N/s)^2 calls
    want = ROUNDS * sum((j["N"] // j["s"]) ** 2 + 1 for j in work)
    assert tcu.tcu_calls() == want
