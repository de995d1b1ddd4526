"""Pins of the oracle's query-independent tier-1 selector (Sec. 4.1, the sigma
equation; Corollary (Ranking stationarity)) against what the mathematics fixes:
a library FFT, closed forms of the low-pass projection, its symmetries, and
brute-force ordering.  CPU only."""
import math

import numpy as np
import pytest

rng = np.random.default_rng(20260904)


def bits(x: np.ndarray) -> np.ndarray:
    """fp32 values -> bf16 bits by truncation (exact for bf16-representable x)."""
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def rand_branch(n: int) -> np.ndarray:
    return bits(rng.standard_normal((n, 64)).astype(np.float32))


@pytest.mark.parametrize("n,kappa", [(4096, 16), (4096, 64), (4096, 1), (4096, 2048), (64, 32), (256, 7)])
def test_sigma_equals_the_library_fft_lowpass(oracle_mod, n, kappa):
    """The DFT sums against numpy's rfft / irfft with bins >= kappa zeroed."""
    r = rand_branch(n)
    x = oracle_mod.decode_bf16(r)
    X = np.fft.rfft(x, axis=0)
    X[kappa:] = 0
    L = np.fft.irfft(X, n=n, axis=0)
    want = np.linalg.norm(x - L, axis=1)
    got = oracle_mod.lowpass_residual_norm(r, kappa)
    assert np.max(np.abs(got - want)) < 1e-12 * np.max(want)


@pytest.mark.parametrize("kappa", [1, 16, 64, 300])
def test_sigma_of_an_impulse_is_the_dirichlet_kernel(oracle_mod, kappa):
    """A unit impulse at row t0 in one channel: the low-pass reconstruction is
    the Dirichlet kernel D(d) / N, D(d) = sin((2 kappa - 1) pi d / N) / sin(pi d / N),
    so sigma_t0 = 1 - (2 kappa - 1) / N and sigma_t = |D(t - t0)| / N elsewhere."""
    N, t0 = 4096, 1234
    x = np.zeros((N, 64), np.float32)
    x[t0, 5] = 1.0
    got = oracle_mod.lowpass_residual_norm(bits(x), kappa)
    d = np.arange(N) - t0
    with np.errstate(invalid="ignore", divide="ignore"):
        D = np.sin((2 * kappa - 1) * np.pi * d / N) / np.sin(np.pi * d / N)
    want = np.abs(D) / N
    want[t0] = 1.0 - (2 * kappa - 1) / N
    assert np.max(np.abs(got - want)) < 1e-13


def test_sigma_of_exact_periodic_signals(oracle_mod):
    """DC is kept whole (sigma = 0); the period-4 wave 1, 0, -1, 0 sits at bin
    N/4, so it is all residual for kappa <= N/4 and none of it for
    kappa > N/4; the period-2 wave (the Nyquist bin) is never kept."""
    N = 4096
    t = np.arange(N)
    dc = np.full((N, 64), 0.75, np.float32)
    assert np.max(oracle_mod.lowpass_residual_norm(bits(dc), 1)) < 1e-13
    q = np.zeros((N, 64), np.float32)
    q[:, 7] = np.choose(t % 4, [1.0, 0.0, -1.0, 0.0])
    s = oracle_mod.lowpass_residual_norm(bits(q), N // 4)
    assert np.max(np.abs(s - np.abs(q[:, 7]))) < 1e-12
    assert np.max(oracle_mod.lowpass_residual_norm(bits(q), N // 4 + 1)) < 1e-12
    ny = np.zeros((N, 64), np.float32)
    ny[:, :4] = np.where(t % 2 == 0, 1.0, -1.0)[:, None]
    s = oracle_mod.lowpass_residual_norm(bits(ny), N // 2)
    assert np.max(np.abs(s - 2.0)) < 1e-12


def test_sigma_parseval(oracle_mod):
    """sum_t sigma_t^2 = sum_c ||x_c||^2 - (|X_0|^2 + 2 sum_{0<f<kappa} |X_f|^2) / N
    (the residual of an orthogonal projection; X from the library FFT)."""
    N, kappa = 4096, 16
    r = rand_branch(N)
    x = oracle_mod.decode_bf16(r)
    X = np.fft.rfft(x, axis=0)
    kept = (np.abs(X[0]) ** 2 + 2 * np.sum(np.abs(X[1:kappa]) ** 2, axis=0)) / N
    want = np.sum(x ** 2) - np.sum(kept)
    got = np.sum(oracle_mod.lowpass_residual_norm(r, kappa) ** 2)
    assert abs(got - want) < 1e-10 * want


def test_sigma_symmetries(oracle_mod):
    """Circular shift along the block shifts sigma (the transform is circular);
    permuting or negating channels leaves it unchanged; a low-pass component
    added to the signal changes nothing."""
    N, kappa = 4096, 16
    r = rand_branch(N)
    s = oracle_mod.lowpass_residual_norm(r, kappa)
    assert np.max(np.abs(oracle_mod.lowpass_residual_norm(np.roll(r, 777, axis=0), kappa)
                         - np.roll(s, 777))) < 1e-12
    perm = rng.permutation(64)
    neg = r[:, perm] ^ np.uint16(0x8000)
    assert np.max(np.abs(oracle_mod.lowpass_residual_norm(neg, kappa) - s)) < 1e-12
    xi = rng.integers(-8, 9, (N, 64)) / 8.0          # exact in bf16, and so is xi + 1
    s1 = oracle_mod.lowpass_residual_norm(bits(xi), kappa)
    s2 = oracle_mod.lowpass_residual_norm(bits(xi + 1.0), kappa)
    assert np.max(np.abs(s1 - s2)) < 1e-12


def test_sigma_close_is_blockwise(oracle_mod):
    """Each closed block is transformed on its own: closing 3 blocks equals the
    three blocks' sigma side by side, and rows past the close are ignored."""
    T = 3 * 512 + 100
    cache = np.zeros((T, 576), np.uint16)
    cache[:, 512:] = rand_branch(T)
    got = oracle_mod.sigma_close(cache, 3 * 512, 8, block=512)
    for b in range(3):
        want = oracle_mod.lowpass_residual_norm(cache[b * 512:(b + 1) * 512, 512:], 8)
        assert np.array_equal(got[b * 512:(b + 1) * 512], want)
    with pytest.raises(ValueError):
        oracle_mod.sigma_close(cache, 700, 8, block=512)


def _brute_tier(sigma, m, nsink):
    n = len(sigma)
    rest = sorted(range(min(nsink, n), n), key=lambda u: (-sigma[u], u))
    return sorted(list(range(min(nsink, n))) + rest[:m])


@pytest.mark.parametrize("n,m,nsink", [(40, 10, 4), (40, 0, 4), (40, 36, 4), (40, 100, 4), (3, 5, 4), (50, 7, 0)])
def test_sigma_select_brute_force_with_ties(oracle_mod, n, m, nsink):
    sigma = rng.integers(0, 6, n).astype(np.float64)      # many exact ties
    got = oracle_mod.sigma_select(sigma, m, nsink)
    assert got.dtype == np.int32
    assert list(got) == _brute_tier(sigma, m, nsink)


def test_blockwise_rebalance_equals_one_shot(oracle_mod):
    """Corollary (Ranking stationarity): the tier kept incrementally as blocks
    close equals the one-shot top-m over the rows closed so far, after every
    close (sigma with planted ties across blocks)."""
    block, nb, m = 64, 9, 50
    sigma = rng.integers(0, 40, block * nb).astype(np.float64)
    sigma[rng.choice(block * nb, 100)] = 17.0
    tiers = oracle_mod.sigma_select_incremental(sigma, m, 4, block=block)
    assert len(tiers) == nb
    for j, tier in enumerate(tiers):
        assert np.array_equal(tier, oracle_mod.sigma_select(sigma[:(j + 1) * block], m, 4))


def test_sigma_finds_planted_anomalies(oracle_mod):
    """Rows whose branch jumps away from a smooth trajectory have the largest
    sigma (what the selector is for): a slowly varying block plus 12 rows with
    an added unit spike in several channels; the top-12 are exactly those."""
    N, kappa = 4096, 16
    t = np.arange(N)[:, None]
    ch = np.arange(64)[None, :]
    smooth = np.cos(2 * np.pi * (1 + ch % 5) * t / N + ch)
    x = smooth.copy()
    spikes = np.sort(rng.choice(np.arange(8, N), 12, replace=False))
    x[spikes, :16] += 1.5
    sigma = oracle_mod.lowpass_residual_norm(bits(x.astype(np.float32)), kappa)
    tier = oracle_mod.sigma_select(sigma, 12, 4)
    assert np.array_equal(tier[4:], spikes)
    assert math.isclose(float(np.min(sigma[spikes])), 1.5 * 4 * (1 - (2 * kappa - 1) / N), rel_tol=0.05)
