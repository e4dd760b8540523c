"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the method: it only draws random matrices
(and a few structured ones: identity, permutation, small integers) on the host
and stores them in the dtype the tensor unit reads.  Both the GPU path and the
CPU oracle are fed the *same bytes* produced here.

Recipe (the paper has no datasets; every input is i.i.d. synthetic):
  * a torch CPU ``Generator`` seeded with the workload's seed draws A first,
    then B;
  * floating-point matrices are drawn in float32 -- uniform on [-1, 1) as
    ``2*rand - 1`` or standard normal -- and rounded once, to nearest-even,
    to float16 / bfloat16;
  * int8 matrices are drawn uniformly from {-128, ..., 127}.
"""
from __future__ import annotations

import torch

# Workloads of the hot path.  "tall": one native call, A (n x s) times
# B (s x s).  "gemm": the blocked N x N product, unit size s.
WORKLOADS = {
    "tall_f16_n4096_s16": dict(kind="tall", dtype="f16", out="f32", n=4096, s=16,
                               dist="uniform", seed=0),
    "gemm_f16_N1024_s16": dict(kind="gemm", dtype="f16", out="f32", N=1024, s=16,
                               dist="uniform", seed=1),
    "gemm_bf16_N8192_s32": dict(kind="gemm", dtype="bf16", out="f32", N=8192, s=32,
                                dist="normal", seed=2),
    "gemm_i8_N8192_s32": dict(kind="gemm", dtype="i8", out="i32", N=8192, s=32,
                              dist="int8", seed=3),
    "tall_bf16_n16777216_s32": dict(kind="tall", dtype="bf16", out="bf16", n=1 << 24,
                                    s=32, dist="normal", seed=4),
}

# Workloads of the rectangular / accumulating product (tcu_gemm_rect):
# C (M x N) [+]= A (M x K) * B (K x N).  Corollary 1's sqrt(n) x r times
# r x sqrt(n) with r below and above sqrt(n), and a product whose order is
# not a multiple of the unit (zero padding).  "acc": accumulate into a
# seeded initial C.
RECT_WORKLOADS = {
    "cor1_bf16_M8192_K2048_N8192_acc": dict(kind="rect", dtype="bf16", out="f32", M=8192,
                                            K=2048, N=8192, s=32, acc=True, dist="normal",
                                            seed=5),
    "cor1_i8_M2048_K65536_N2048_acc": dict(kind="rect", dtype="i8", out="i32", M=2048,
                                           K=65536, N=2048, s=32, acc=True, dist="int8",
                                           seed=6),
    "pad_bf16_M8200_K8200_N8200": dict(kind="rect", dtype="bf16", out="bf16", M=8200, K=8200,
                                       N=8200, s=32, acc=False, dist="normal", seed=7),
}

# Workloads of batch polynomial evaluation (tcu_poly_eval, Theorem 11):
# n coefficients ~ N(0,1) and p points ~ U[-1, 1), both in the input type.
POLY_WORKLOADS = {
    "poly_bf16_n4096_p16777216_s32": dict(kind="poly", dtype="bf16", out="f32", n=4096,
                                          p=1 << 24, s=32, seed=8),
    # a long polynomial: n/m = 64 unit calls per point, where the theorem's
    # matrix term n p / sqrt(m) dominates its scalar terms
    "poly_bf16_n65536_p4194304_s32": dict(kind="poly", dtype="bf16", out="f32", n=1 << 16,
                                          p=1 << 22, s=32, seed=11),
}

# Workloads of the transitive closure (tcu_transitive_closure, Theorem 5):
# a random digraph of n vertices, each ordered pair an edge with probability
# deg / n (mean out-degree deg).
TC_WORKLOADS = {
    "tc_n8192_deg2": dict(kind="tc", n=8192, deg=2.0, s=32, seed=9),
}

# Workloads of the DFT (tcu_dft, Theorem 7): batch complex64 vectors of
# length n, real and imaginary parts ~ N(0, 1).
DFT_WORKLOADS = {
    "dft_c64_n1048576_b16_s32": dict(kind="dft", n=1 << 20, batch=16, s=32, seed=10),
}

TORCH_DTYPE = {"f16": torch.float16, "bf16": torch.bfloat16, "i8": torch.int8,
               "f32": torch.float32, "i32": torch.int32}


def draw(shape, dtype: str, dist: str, gen: torch.Generator) -> torch.Tensor:
    """One random matrix in storage dtype ``dtype`` ('f16', 'bf16', 'i8')."""
    if dtype == "i8":
        if dist not in ("int8", "uniform"):
            raise ValueError(f"int8 inputs are drawn uniformly, not {dist!r}")
        return torch.randint(-128, 128, shape, generator=gen, dtype=torch.int8)
    if dist == "uniform":
        x = torch.rand(shape, generator=gen, dtype=torch.float32).mul_(2.0).sub_(1.0)
    elif dist == "normal":
        x = torch.randn(shape, generator=gen, dtype=torch.float32)
    elif dist == "smallint":
        x = torch.randint(-2, 3, shape, generator=gen).to(torch.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return x.to(TORCH_DTYPE[dtype])


def draw_on(device, shape, dtype: str, dist: str, seed: int) -> torch.Tensor:
    """As ``draw`` with torch's own generator on ``device`` (seeded): for
    inputs too large to draw on the host and copy.  The oracle is given the
    same stored bytes, copied back."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    if dtype == "i8":
        return torch.randint(-128, 128, shape, generator=gen, dtype=torch.int8, device=device)
    if dist == "uniform":
        x = torch.rand(shape, generator=gen, dtype=torch.float32, device=device).mul_(2.0).sub_(1.0)
    elif dist == "normal":
        x = torch.randn(shape, generator=gen, dtype=torch.float32, device=device)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return x.to(TORCH_DTYPE[dtype])


def cycle_graph(n: int, max_len: int, seed: int):
    """A directed graph on n vertices that is a disjoint union of cycles: the
    vertices in a random order, cut at random points into runs of 1 ..
    max_len vertices, each run closed into a cycle (a run of one vertex is a
    self loop).  Returns (src, dst, label) as int64 tensors: the edges, and
    for every vertex the index of its cycle."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    order = torch.randperm(n, generator=gen)
    lens = torch.randint(1, max_len + 1, (n,), generator=gen)
    ends = torch.cumsum(lens, 0)
    ends = ends[ends < n]
    starts = torch.cat([torch.zeros(1, dtype=torch.int64), ends])
    stops = torch.cat([ends, torch.tensor([n])])
    src, dst = [], []
    label = torch.empty(n, dtype=torch.int64)
    for c, (a, b) in enumerate(zip(starts.tolist(), stops.tolist())):
        run = order[a:b]
        src.append(run)
        dst.append(torch.roll(run, -1))
        label[run] = c
    return torch.cat(src), torch.cat(dst), label


def shapes(spec: dict):
    """(A shape, B shape, C shape) of a workload spec."""
    if spec["kind"] == "tall":
        n, s = spec["n"], spec["s"]
        return (n, s), (s, s), (n, s)
    if spec["kind"] == "rect":
        M, K, N = spec["M"], spec["K"], spec["N"]
        return (M, K), (K, N), (M, N)
    N = spec["N"]
    return (N, N), (N, N), (N, N)


def make_inputs(spec: dict, seed: int | None = None):
    """Draw (A, B) on the host for a workload spec: A first, then B."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(spec["seed"] if seed is None else seed)
    a_shape, b_shape, _ = shapes(spec)
    A = draw(a_shape, spec["dtype"], spec["dist"], gen)
    B = draw(b_shape, spec["dtype"], spec["dist"], gen)
    return A, B


def make_poly_inputs(spec: dict):
    """(coefficients, points) of a polynomial workload: coefficients first."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(spec["seed"])
    coef = draw((spec["n"],), spec["dtype"], "normal", gen)
    pts = draw((spec["p"],), spec["dtype"], "uniform", gen)
    return coef, pts


def digraph(n: int, avg_out_degree: float, seed: int) -> torch.Tensor:
    """Random directed graph as an n x n int8 0/1 adjacency matrix: each
    ordered pair (i, j), self loops included, is an edge independently with
    probability avg_out_degree / n."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    q = min(1.0, avg_out_degree / max(n, 1))
    return (torch.rand((n, n), generator=gen) < q).to(torch.int8)


def make_tc_input(spec: dict) -> torch.Tensor:
    """Adjacency matrix (int8 0/1) of a transitive-closure workload."""
    return digraph(spec["n"], spec["deg"], spec["seed"])


def complex_signal(batch: int, n: int, seed: int) -> torch.Tensor:
    """batch x n complex64 values, real and imaginary parts ~ N(0, 1), drawn
    as one (batch, n, 2) float32 array."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    return torch.view_as_complex(torch.randn((batch, n, 2), generator=gen, dtype=torch.float32))


def make_c0(spec: dict) -> torch.Tensor:
    """Initial output of an accumulating workload: standard normal in the
    output type (float32 or bfloat16), or int32 uniform in [-2^20, 2^20),
    from its own generator seeded with the workload's seed + 1000."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(spec["seed"] + 1000)
    _, _, c_shape = shapes(spec)
    if spec["out"] == "i32":
        return torch.randint(-(1 << 20), 1 << 20, c_shape, generator=gen, dtype=torch.int32)
    return torch.randn(c_shape, generator=gen, dtype=torch.float32).to(TORCH_DTYPE[spec["out"]])


def small_ints(shape, dtype: str, seed: int) -> torch.Tensor:
    """Integers in {-2..2} stored in ``dtype`` (exact in every storage type)."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    return torch.randint(-2, 3, shape, generator=gen).to(TORCH_DTYPE[dtype])


def identity(s: int, dtype: str) -> torch.Tensor:
    return torch.eye(s, dtype=torch.float32).to(TORCH_DTYPE[dtype])


def permutation(s: int, dtype: str, seed: int):
    """(P, perm) with P[perm[j], j] = 1, so (A P)[:, j] = A[:, perm[j]]."""
    gen = torch.Generator(device="cpu")
    gen.manual_seed(seed)
    perm = torch.randperm(s, generator=gen)
    P = torch.zeros(s, s, dtype=torch.float32)
    P[perm, torch.arange(s)] = 1.0
    return P.to(TORCH_DTYPE[dtype]), perm


def bits(t: torch.Tensor):
    """Stored bytes of a CPU tensor as a numpy array (uint16 for 16-bit
    floats, int8 for int8) -- the form the oracle reads."""
    import numpy as np
    t = t.contiguous()
    if t.dtype in (torch.float16, torch.bfloat16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.int8:
        return t.numpy()
    raise TypeError(f"no stored-bits view for {t.dtype}")
