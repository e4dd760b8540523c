"""The allocation-free DFT (tcu_dft_noalloc), through the C ABI: its output
equals tcu_dft's (with a caller work buffer) on the same inputs, and both
meet the oracle's bar (the definition on sampled outputs), on two calls in a
row -- the second on a smaller input, so it runs on the scratch the first
call left behind -- plus the size limit and a one-level transform."""
import numpy as np
import pytest
import torch

from oracle import compare
from paper_1908_06649_amd import inputs, tcu

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _noalloc(x: torch.Tensor, s: int) -> np.ndarray:
    batch, n = x.shape
    dx = x.to(DEV).contiguous()
    guard = 1024
    ybuf = torch.full((batch * n + guard,), complex(7.0, -7.0), dtype=torch.complex64,
                      device=DEV)
    y = ybuf[: batch * n]
    st = torch.cuda.current_stream().cuda_stream
    rc = tcu.lib().tcu_dft_noalloc(dx.data_ptr(), y.data_ptr(), n, batch, s, st)
    assert rc == tcu.TCU_OK, tcu.tcu_strerror(rc)
    torch.cuda.synchronize()
    assert bool((ybuf[batch * n:] == complex(7.0, -7.0)).all()), "wrote past y"
    assert torch.equal(dx.cpu(), x), "x changed"
    return y.view(batch, n).cpu().numpy()


def _with_work(x: torch.Tensor, s: int) -> np.ndarray:
    batch, n = x.shape
    dx = x.to(DEV).contiguous()
    y = torch.empty(batch * n, dtype=torch.complex64, device=DEV)
    work = torch.empty_like(y)
    tcu.tcu_set_unit(s)
    tcu.tcu_dft(dx, y, work, n, batch)
    torch.cuda.synchronize()
    return y.view(batch, n).cpu().numpy()


@pytest.mark.parametrize("s", [32, 16])
def test_noalloc_matches_dft_two_calls(s):
    # first call: the whole scratch (8 vectors of 2^20 = 64 MiB), then a
    # smaller one (3 vectors of 2^13) on what the first left behind
    for batch, n, seed in ((8, 1 << 20, 71), (3, 1 << 13, 72)):
        assert batch * n * 8 <= tcu.TCU_DFT_NOALLOC_MAX_BYTES
        x = inputs.complex_signal(batch, n, seed + s)
        tcu.tcu_reset_calls()
        got = _noalloc(x, s)
        calls = tcu.tcu_calls()
        ref = _with_work(x, s)
        assert tcu.tcu_calls() == 2 * calls          # counted as tcu_dft counts
        assert np.array_equal(got, ref), "differs from tcu_dft"
        rep = compare.check_dft(x.numpy(), got)
        print(s, batch, n, rep)


def test_noalloc_size_limit_and_one_level():
    n = 1 << 20
    x = torch.zeros(9 * n, dtype=torch.complex64, device=DEV)
    y = torch.full((9 * n,), complex(3.0, 3.0), dtype=torch.complex64, device=DEV)
    st = torch.cuda.current_stream().cuda_stream
    tcu.tcu_reset_calls()
    rc = tcu.lib().tcu_dft_noalloc(x.data_ptr(), y.data_ptr(), n, 9, 32, st)
    assert rc == tcu.TCU_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((y == complex(3.0, 3.0)).all()) and tcu.tcu_calls() == 0
    # one level (n <= s) needs no scratch: any batch
    xs = inputs.complex_signal(1 << 19, 32, 73)
    got = _noalloc(xs, 32)
    assert np.array_equal(got, _with_work(xs, 32))
