"""Pins of the oracle's DFT (Section 4.5) against what the mathematics fixes
(CPU only).

dft_direct is the definition y[k] = sum_j x[j] exp(-2 pi i j k / n).  It is
checked against closed-form transforms (a unit impulse, a constant, a pure
complex exponential, a cosine, a shifted impulse), Parseval's identity,
linearity, the circular shift theorem and the transform of the conjugate,
and against exact rational arithmetic on sizes where the twiddles are exact
(n = 1, 2, 4: W entries in {+-1, +-i}).  numpy's FFT (oracle.dft, used at
large sizes) is checked against dft_direct.  dft_direct_at (the definition
at chosen outputs, for vectors too long for the whole O(n^2) transform)
equals dft_direct's entries and meets the closed forms at n = 2^16, 2^20.  Plausible mistakes (the
conjugate sign, the transpose of a non-symmetric use, an off-by-one
frequency) fail the pins.
"""
import numpy as np
import pytest

import oracle

RNG = np.random.default_rng(42)


def rand_c(shape):
    return RNG.standard_normal(shape) + 1j * RNG.standard_normal(shape)


@pytest.mark.parametrize("n", [1, 2, 3, 8, 17, 64, 100])
def test_dft_closed_forms(n):
    delta = np.zeros(n, complex)
    delta[0] = 1
    assert np.allclose(oracle.dft_direct(delta), np.ones(n), atol=1e-14)
    assert np.allclose(oracle.dft_direct(np.ones(n, complex)),
                       np.eye(1, n, 0).ravel() * n, atol=1e-10)
    for f in range(min(n, 5)):
        e = np.exp(2j * np.pi * f * np.arange(n) / n)        # exp(+2 pi i f j / n)
        want = np.zeros(n, complex)
        want[f] = n
        assert np.allclose(oracle.dft_direct(e), want, atol=1e-9 * n)
    if n > 2:
        c = np.cos(2 * np.pi * 1 * np.arange(n) / n)
        want = np.zeros(n, complex)
        want[1] += n / 2
        want[n - 1] += n / 2
        assert np.allclose(oracle.dft_direct(c), want, atol=1e-9 * n)
        shifted = np.zeros(n, complex)
        shifted[2] = 1                                          # x = delta[j - 2]
        assert np.allclose(oracle.dft_direct(shifted),
                           np.exp(-2j * np.pi * 2 * np.arange(n) / n), atol=1e-12)


@pytest.mark.parametrize("n", [1, 2, 4])
def test_dft_exact_small(n):
    """For n <= 4 every entry of W is +-1 or +-i: against that matrix, written
    out by hand, on small integers (the definition's binary64 cos/sin of
    pi and pi/2 are off by at most 2^-53 of a unit)."""
    x = RNG.integers(-5, 6, (6, n)) + 1j * RNG.integers(-5, 6, (6, n))
    w = np.array([[1, 1, 1, 1], [1, -1j, -1, 1j], [1, -1, 1, -1], [1, 1j, -1, -1j]])[:n, :n]
    if n == 2:
        w = np.array([[1, 1], [1, -1]])
    want = x @ w
    mag = np.sum(np.abs(x), axis=1, keepdims=True)
    assert np.all(np.abs(oracle.dft_direct(x) - want) <= 4 * 2.0 ** -52 * mag)


def test_dft_identities():
    n = 96
    x, z = rand_c((4, n)), rand_c((4, n))
    X, Z = oracle.dft_direct(x), oracle.dft_direct(z)
    assert np.allclose(np.sum(np.abs(X) ** 2, axis=1), n * np.sum(np.abs(x) ** 2, axis=1))
    assert np.allclose(oracle.dft_direct(2.5 * x - 1j * z), 2.5 * X - 1j * Z)
    m = 7
    xs = np.roll(x, m, axis=1)                                   # x[j - m]
    assert np.allclose(oracle.dft_direct(xs), X * np.exp(-2j * np.pi * m * np.arange(n) / n))
    # DFT(conj(x))[k] = conj(DFT(x)[-k])
    assert np.allclose(oracle.dft_direct(np.conj(x)), np.conj(np.roll(X[:, ::-1], 1, axis=1)))


@pytest.mark.parametrize("n", [2, 32, 256, 2048])
def test_fft_matches_definition(n):
    x = rand_c((3, n))
    d, f = oracle.dft_direct(x), oracle.dft(x)
    assert np.max(np.abs(d - f)) <= 1e-9 * np.sum(np.abs(x), axis=1).max()


@pytest.mark.parametrize("n", [1, 3, 64, 100, 2048])
def test_sampled_definition_equals_full(n):
    """dft_direct_at is the definition at chosen outputs: equal to the whole
    transform's entries (same binary64 evaluation order)."""
    x = rand_c((3, n))
    ks = np.unique(np.concatenate([[0, n // 2, n - 1], RNG.integers(0, n, 9)]))
    assert np.array_equal(oracle.dft_direct_at(x, ks), oracle.dft_direct(x)[:, ks])
    assert np.array_equal(oracle.dft_direct_at(x[0], ks), oracle.dft_direct(x[0])[ks])


@pytest.mark.parametrize("n", [1 << 16, 1 << 20])
def test_sampled_definition_closed_forms_large(n):
    """At sizes where the whole definition is too slow, the sampled outputs
    against closed forms: a shifted impulse delta[j - m] (y[k] = w^(mk),
    exercising the exact reduction of m k mod n), and a pure exponential of
    frequency f (y[k] = n at k = f, 0 elsewhere)."""
    from oracle import compare
    ks = compare.dft_sample_freqs(n, seed=5)
    assert ks.size >= 72 and {0, 1, n // 2, n - 1} <= set(ks.tolist())
    m = 12345
    x = np.zeros(n, complex)
    x[m] = 1
    want = np.exp(-2j * np.pi * ((m * ks) % n) / n)
    assert np.max(np.abs(oracle.dft_direct_at(x, ks) - want)) <= 1e-12
    f = int(ks[len(ks) // 2])
    e = np.exp(2j * np.pi * ((f * np.arange(n)) % n) / n)
    want = np.where(ks == f, n, 0)
    assert np.max(np.abs(oracle.dft_direct_at(e, ks) - want)) <= 1e-9 * n


def test_sampled_definition_matches_fft_large():
    """The sampled definition against numpy's FFT on random data, n = 2^14."""
    from oracle import compare
    n = 1 << 14
    x = rand_c((2, n))
    ks = compare.dft_sample_freqs(n, seed=7)
    d = oracle.dft_direct_at(x, ks)
    f = oracle.dft(x)[:, ks]
    assert np.max(np.abs(d - f)) <= 1e-9 * np.sum(np.abs(x), axis=1).max()


def test_check_dft_uses_definition_on_large_n():
    """compare.check_dft takes the definition at >= 64 outputs for n > 1024
    and rejects a transform that is wrong at only one of those outputs."""
    from oracle import compare
    n = 4096
    x = rand_c((2, n))
    y = oracle.dft(x)
    rep = compare.check_dft(x, y)
    assert rep["freqs_checked"] >= 72
    ks = compare.dft_sample_freqs(n)
    bad = y.copy()
    bad[1, ks[40]] += 0.05 * np.sum(np.abs(x[1]))
    with pytest.raises(AssertionError):
        compare.check_dft(x, bad, fft_extra=False)


def _mutants():
    def conj_sign(x):
        return np.conj(oracle.dft_direct(np.conj(x)))           # exp(+2 pi i jk/n)

    def off_by_one(x):
        return np.roll(oracle.dft_direct(x), 1, axis=-1)

    def unnormalized_half(x):
        return oracle.dft_direct(x) / 2

    def wrong_base(x):                                          # w = exp(-2 pi i / (n + 1))
        n = x.shape[-1]
        jk = np.outer(np.arange(n), np.arange(n))
        return x @ np.exp(-2j * np.pi * jk / (n + 1))

    return [conj_sign, off_by_one, unnormalized_half, wrong_base]


def test_pins_catch_planted_mistakes():
    n = 8
    shifted = np.zeros(n, complex)
    shifted[2] = 1
    want = np.exp(-2j * np.pi * 2 * np.arange(n) / n)
    for mut in _mutants():
        assert not np.allclose(mut(shifted), want, atol=1e-12), mut.__name__
