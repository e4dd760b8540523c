"""GPU parity of the transitive closure (tcu_transitive_closure, Theorem 5,
Section 4.3) against the CPU oracle, through the C ABI.  Results are 0/1
matrices and must match the oracle exactly (a closure is unique)."""
import numpy as np
import pytest
import torch

import oracle
from paper_1908_06649_amd import inputs, tcu

import gpu_util as gu

pytestmark = pytest.mark.gpu

SENT = 0x5A


def run_tc(d: np.ndarray, ld: int | None = None, s: int = 32) -> np.ndarray:
    """Closure of host adjacency matrix d on the GPU in an array of row pitch
    ld, with a guard region after it; checks that no byte outside the n x n
    view changed."""
    n = d.shape[0]
    ld = n if ld is None else ld
    rows = max(n, 1)
    total = rows * max(ld, 1)
    buf = torch.full((total + 4096,), SENT, dtype=torch.uint8, device=gu.DEV)
    view = buf[:total].view(rows, max(ld, 1))[:n, :n]
    view.copy_(torch.from_numpy(np.ascontiguousarray(d)).to(gu.DEV))
    tcu.tcu_set_unit(s)
    tcu.tcu_transitive_closure(view, n, ld)
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    grid = host[:total].reshape(rows, max(ld, 1))
    assert np.all(grid[:, n:] == SENT), "wrote into the row padding"
    assert np.all(host[total:] == SENT), "wrote past the array"
    return grid[:n, :n].copy()


def graph(n, deg, seed):
    return inputs.digraph(n, deg, seed).numpy().view(np.uint8)


SIZES = [1, 2, 15, 16, 17, 100, 255, 256, 257, 300, 511, 512, 513, 600, 768, 1000, 1024, 1280,
         1500, 2048]


@pytest.mark.parametrize("deg", [0.7, 1.3, 3.0])
@pytest.mark.parametrize("n", SIZES)
def test_tc_random_graphs(n, deg):
    d = graph(n, deg, n * 7 + int(deg * 10))
    assert np.array_equal(run_tc(d), oracle.transitive_closure(d))


# The D update of each band also closes the next band's diagonal block in
# its workgroup 0 while the others take the remaining tiles; with a tiny
# persistent grid every other workgroup walks many tiles around that one
# (grid 2: workgroup 1 takes them all; grid 1: no fused closure).
@pytest.mark.parametrize("grid", [1, 2, 3, 7, 29])
@pytest.mark.parametrize("n", [512, 1280, 2048])
def test_tc_fused_diagonal_small_grids(n, grid, knobs):
    knobs(tcu.TCU_KNOB_PP_GRID, grid)
    d = graph(n, 1.1, n + grid)
    assert np.array_equal(run_tc(d), oracle.transitive_closure(d))


@pytest.mark.parametrize("n,ld", [(300, 304), (300, 301), (513, 528), (700, 777), (1000, 1024)])
def test_tc_pitched(n, ld):
    d = graph(n, 1.2, n + ld)
    assert np.array_equal(run_tc(d, ld), oracle.transitive_closure(d))


@pytest.mark.parametrize("n", [700, 1536, 2000, 2560])
def test_tc_long_paths_cross_every_band(n):
    """A path i -> i+1 (closure: strict upper triangle) and its reverse:
    reachability has to travel through every pivot band."""
    path = np.eye(n, k=1, dtype=np.uint8)
    assert np.array_equal(run_tc(path), np.triu(np.ones((n, n), np.uint8), 1))
    rev = np.ascontiguousarray(path.T)
    assert np.array_equal(run_tc(rev), np.tril(np.ones((n, n), np.uint8), -1))
    perm = np.random.default_rng(n).permutation(n)          # a path in scrambled order
    p = np.zeros((n, n), np.uint8)
    p[perm[:-1], perm[1:]] = 1
    assert np.array_equal(run_tc(p), oracle.transitive_closure(p))


@pytest.mark.parametrize("n", [512, 1024, 1792])
def test_tc_structured_across_bands(n):
    """Graphs whose reachability must cross band boundaries in both
    directions (whole bands: the look-ahead schedule): a few long cycles
    woven through every band, plus a sparse random layer."""
    rng = np.random.default_rng(n)
    d = np.zeros((n, n), np.uint8)
    for _ in range(3):
        perm = rng.permutation(n)[: n // 3]
        d[perm, np.roll(perm, 1)] = 1
    d |= graph(n, 0.3, n + 1)
    assert np.array_equal(run_tc(d), oracle.transitive_closure(d))


def test_tc_cycle_and_empty():
    n = 900
    cyc = np.roll(np.eye(n, dtype=np.uint8), 1, axis=1)
    assert np.all(run_tc(cyc) == 1)
    assert not np.any(run_tc(np.zeros((n, n), np.uint8)))


def test_tc_nonzero_bytes_are_edges():
    """Any nonzero byte (e.g. 5 or 0xFF) is an edge; the output is 0/1."""
    d = graph(400, 1.2, 9)
    vals = np.random.default_rng(2).choice(np.array([1, 5, 0x80, 0xFF], np.uint8), d.shape)
    got = run_tc((d * vals).astype(np.uint8))
    assert np.array_equal(got, oracle.transitive_closure(d))


def test_tc_empty_and_accounting():
    tcu.tcu_reset_calls()
    buf = torch.zeros(16, dtype=torch.uint8, device=gu.DEV)
    tcu.tcu_transitive_closure(buf[:0].view(0, 0), 0, 0)
    assert tcu.tcu_calls() == 0
    n, s = 1000, 32
    run_tc(graph(n, 1.0, 3), s=s)
    q = -(-n // s)
    assert tcu.tcu_calls() == q * (q - 1)


@pytest.mark.parametrize("name", sorted(inputs.TC_WORKLOADS))
def test_tc_workload(name):
    sp = inputs.TC_WORKLOADS[name]
    d = inputs.make_tc_input(sp).numpy().view(np.uint8)
    got = run_tc(d, s=sp["s"])
    want = oracle.transitive_closure(d)
    assert np.array_equal(got, want)
    print(name, "closure density", float(want.mean()))


def test_tc_on_side_stream_joins():
    """On a non-default stream: once the caller's stream is synchronized (and
    nothing else), every update of the closure has landed."""
    n = 2048
    d = graph(n, 1.0, 77)
    want = oracle.transitive_closure(d)
    st = torch.cuda.Stream()
    X = torch.from_numpy(d).to(gu.DEV)
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        tcu.tcu_transitive_closure(X, n, n)
        out = torch.empty((n, n), dtype=torch.uint8, device="cpu", pin_memory=True)
        out.copy_(X, non_blocking=True)
    st.synchronize()
    assert np.array_equal(out.numpy(), want)


def test_tc_two_streams_back_to_back():
    """Two closures enqueued on two streams without a synchronization in
    between (they share the library's second stream and events)."""
    n = 1536
    ds = [graph(n, 1.2, 5), graph(n, 0.8, 6)]
    Xs = [torch.from_numpy(d).to(gu.DEV) for d in ds]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    for X, st in zip(Xs, streams):
        tcu.tcu_transitive_closure_ex(X, n, n, 32, st.cuda_stream)
    torch.cuda.synchronize()
    for X, d in zip(Xs, ds):
        assert np.array_equal(X.cpu().numpy(), oracle.transitive_closure(d))
