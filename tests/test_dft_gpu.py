"""GPU parity of the DFT (tcu_dft, Theorem 7, Section 4.5) against the CPU
oracle, through the C ABI: the definition y[k] = sum_j x[j] w^(jk) on every
output for n <= 1024, and on at least 64 outputs of every vector above
(k = 0, 1, 2, n/2 - 1, n/2, n/2 + 1, n - 2, n - 1 and 64 seeded random
frequencies), with numpy's binary64 FFT of the whole transform as an extra
check.  Bar: relative Frobenius error <= 1e-3 per vector and elementwise
|err_k| <= 1e-2 * sum_j |x_j|."""
import numpy as np
import pytest
import torch

from oracle import compare
from paper_1908_06649_amd import inputs, tcu

import gpu_util as gu

pytestmark = pytest.mark.gpu


def run_dft(x: torch.Tensor, s: int, with_work: bool = True) -> np.ndarray:
    batch, n = x.shape
    dx = x.to(gu.DEV).contiguous()
    guard = 1024
    ybuf = torch.full((batch * n + guard,), complex(7.0, -7.0), dtype=torch.complex64,
                      device=gu.DEV)
    y = ybuf[: batch * n]
    work = (torch.empty(batch * n, dtype=torch.complex64, device=gu.DEV) if with_work else None)
    tcu.tcu_set_unit(s)
    tcu.tcu_dft(dx, y, work, n, batch)
    torch.cuda.synchronize()
    assert bool((ybuf[batch * n:] == complex(7.0, -7.0)).all()), "wrote past y"
    assert torch.equal(dx.cpu(), x), "x changed"
    return y.view(batch, n).cpu().numpy()


# 2^21 and 2^23: levels with N_t above 2^20, whose twiddles are single
# sincospi evaluations rather than products of two table entries
SIZES = [1, 2, 4, 8, 16, 32, 64, 128, 512, 1024, 2048, 4096, 32768, 65536, 1 << 20, 1 << 21,
         1 << 23]


# one vector of 2^20 or more per unit size here; the workload test runs a batch of them
CASES = [(n, b) for n in SIZES for b in (1, 3) if n < 1 << 20 or b == 1]


@pytest.mark.parametrize("s", [16, 32])
@pytest.mark.parametrize("n,batch", CASES)
def test_dft_sizes(n, batch, s):
    x = inputs.complex_signal(batch, n, seed=n + 13 * batch + s)
    got = run_dft(x, s, with_work=True)
    rep = compare.check_dft(x.numpy(), got)
    assert rep["max_rel_frob"] <= 1e-4, rep      # the hi/lo products keep ~2^-16 per level


@pytest.mark.parametrize("s", [16, 32])
def test_dft_closed_forms(s):
    n = 4096
    x = torch.zeros(3, n, dtype=torch.complex64)
    x[0, 0] = 1                                          # impulse -> all ones
    x[1, :] = 1                                          # constant -> n at k = 0
    j = torch.arange(n, dtype=torch.float64)
    x[2] = torch.polar(torch.ones(n, dtype=torch.float64), 2 * np.pi * 5 * j / n).to(torch.complex64)
    got = run_dft(x, s)
    assert np.allclose(got[0], 1, atol=1e-5)
    want = np.zeros(n, complex)
    want[0] = n
    assert np.allclose(got[1], want, atol=1e-3)
    want = np.zeros(n, complex)
    want[5] = n
    assert np.allclose(got[2], want, atol=2e-2)


def test_dft_single_level_needs_no_work():
    x = inputs.complex_signal(4, 32, seed=3)
    compare.check_dft(x.numpy(), run_dft(x, 32, with_work=False))


def test_dft_empty_batch_and_accounting():
    tcu.tcu_reset_calls()
    e = torch.empty(0, dtype=torch.complex64, device=gu.DEV)
    tcu.tcu_dft(e, e.clone(), e.clone(), 1024, 0)
    assert tcu.tcu_calls() == 0
    n, s, batch = 65536, 32, 2
    run_dft(inputs.complex_signal(batch, n, 1), s)
    # 65536 = 2^16 with s = 32: levels of radix 32, 32, 32 and 2
    assert tcu.tcu_calls() == 4 * batch * 4


def test_dft_deterministic():
    x = inputs.complex_signal(2, 32768, seed=4)
    assert np.array_equal(run_dft(x, 32), run_dft(x, 32))


@pytest.mark.parametrize("name", sorted(inputs.DFT_WORKLOADS))
def test_dft_workload(name):
    sp = inputs.DFT_WORKLOADS[name]
    x = inputs.complex_signal(sp["batch"], sp["n"], sp["seed"])
    got = run_dft(x, sp["s"])
    rep = compare.check_dft(x.numpy(), got)
    assert rep["freqs_checked"] >= 64
    print(name, rep)


# Sizes where two consecutive full-radix levels run as one launch: for s = 32
# the first two levels from n = 2^14 (16 groups J' per vector) and levels 3-4
# at n = 2^20 (P = 2^10); for s = 16 from n = 2^12, and levels 2-3 at
# n = 2^16 (P = 16).  At n = 2^21 (s = 32) and 2^22 (s = 16) the first
# level's N_t is above 2^20 (twiddles by sincospi) and the second's below
# (twiddles from the tables).
PAIR_CASES = [(1 << 12, 3, 16), (1 << 14, 2, 16), (1 << 16, 2, 16), (1 << 14, 3, 32),
              (1 << 15, 2, 32), (1 << 20, 2, 32), (1 << 18, 1, 16), (1 << 21, 1, 32),
              (1 << 22, 1, 16)]


@pytest.mark.parametrize("n,batch,s", PAIR_CASES)
def test_dft_level_pairs_bit_identical(knobs, n, batch, s):
    """Two levels in one launch (the default where possible) give the same
    bits as one launch per level (TCU_KNOB_DFT_PAIRS = 1): every value takes
    the same operations either way."""
    x = inputs.complex_signal(batch, n, seed=n + 7 * batch + s)
    paired = run_dft(x, s)
    knobs(tcu.TCU_KNOB_DFT_PAIRS, 1)
    single = run_dft(x, s)
    assert np.array_equal(paired.view(np.uint64), single.view(np.uint64))
    rep = compare.check_dft(x.numpy(), paired)
    assert rep["max_rel_frob"] <= 1e-4, rep
