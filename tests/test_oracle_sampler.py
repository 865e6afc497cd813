"""Pin the oracle's sampling distribution (O5) and inverse-CDF draw (O6) with exact
arithmetic, brute force and a chi-square test on the real random stream."""
import math
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import oracle


def _rho(d, seed=0):
    return np.abs(np.random.default_rng(seed).standard_normal(d)).astype(np.float32) + np.float32(0.1)


def test_fixed_point_weights_exact():
    rng = np.random.default_rng(1)
    for trial in range(20):
        d = int(rng.integers(1, 300))
        x = (rng.standard_normal(d) * 10.0 ** rng.integers(-30, 30)).astype(np.float32)
        x[rng.random(d) < 0.2] = 0
        rho = _rho(d, trial)
        fp = oracle.fixed_point_weights(x, rho)
        if not np.any(x):
            assert fp is None
            continue
        w, C, T = fp
        v = [Fraction(float(np.float32(abs(np.float32(a)) * b))) for a, b in zip(x, rho)]
        vmax = max(v)
        # exponent e with vmax in [2^(e-1), 2^e)
        e = math.floor(math.log2(vmax)) + 1
        while Fraction(2) ** (e - 1) > vmax:
            e -= 1
        while vmax >= Fraction(2) ** e:
            e += 1
        ref = [math.floor(vi * Fraction(2) ** (32 - e)) for vi in v]
        assert w == ref
        assert 2 ** 31 <= max(w) < 2 ** 32
        assert C[-1] == T == sum(w) and all(C[i] <= C[i + 1] for i in range(d - 1))


def test_subnormal_products():
    x = np.array([1e-25, -2e-25, 0.0, 3e-26], np.float32)
    rho = np.array([1e-15, 1e-15, 1.0, 1e-15], np.float32)
    v = np.abs(x) * rho
    assert np.all(v[[0, 1, 3]] > 0) and np.all(v[[0, 1, 3]] < np.finfo(np.float32).tiny)
    w, C, T = oracle.fixed_point_weights(x, rho)
    assert w[2] == 0 and w[1] >= 2 ** 31 and w[0] > 0 and w[3] > 0


def test_scale_equivariance_same_indices():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(96).astype(np.float32)
    rho = _rho(96)
    w0, C0, T0 = oracle.fixed_point_weights(x, rho)
    for k in (-40, -3, 5, 60):
        w, C, T = oracle.fixed_point_weights((x * np.float32(2.0 ** k)).astype(np.float32), rho)
        assert w == w0
        assert oracle.draw_indices(C, T, 50, 9, 0, 3) == oracle.draw_indices(C0, T0, 50, 9, 0, 3)


def test_equal_weights_uniform():
    x = np.full(64, -1.5, np.float32)
    rho = np.full(64, 0.75, np.float32)
    w, C, T = oracle.fixed_point_weights(x, rho)
    assert len(set(w)) == 1 and T == 64 * w[0]


def test_inverse_cdf_brute_force():
    # every t in [0, T) maps to index i exactly w_i times; zero-weight rows never
    w = [3, 0, 5, 2, 0, 0, 1, 4]
    C = [int(c) for c in np.cumsum(w)]
    T = C[-1]
    hits = [0] * len(w)
    for t in range(T):
        # u chosen so that floor(u T / 2^64) = t exactly: u = ceil(t 2^64 / T)
        u = -((-t << 64) // T)
        assert (u * T) >> 64 == t
        hits[oracle.index_from_u(u, C, T)] += 1
    assert hits == w


def test_u64_mass_exact():
    # the u in [0, 2^64) that map to index i form [ceil(C_{i-1} 2^64/T), ceil(C_i 2^64/T))
    rng = np.random.default_rng(5)
    w = [int(v) for v in rng.integers(0, 2 ** 32, size=40)]
    w[7] = 0
    w[8] = 0
    C = [int(c) for c in np.cumsum(np.array(w, dtype=object))]
    T = C[-1]
    lo = 0
    for i, wi in enumerate(w):
        hi = -((-C[i] << 64) // T)
        if wi == 0:
            assert hi == lo
            continue
        assert hi > lo
        assert oracle.index_from_u(lo, C, T) == i
        assert oracle.index_from_u(hi - 1, C, T) == i
        lo = hi
    assert lo == 1 << 64
    assert oracle.index_from_u((1 << 64) - 1, C, T) == len(w) - 1


def test_draws_chi_square():
    rng = np.random.default_rng(6)
    x = rng.standard_normal(48).astype(np.float32)
    rho = _rho(48, 6)
    w, C, T = oracle.fixed_point_weights(x, rho)
    idx = oracle.draw_indices(C, T, 200_000, 12345, 3, 17)
    counts = np.bincount(idx, minlength=48)
    expected = np.array(w, dtype=np.float64) / T * len(idx)
    chi2, p = stats.chisquare(counts, expected)
    assert p > 1e-4, (chi2, p)


def test_draw_prefix_property():
    # draw k does not depend on r: r and r+1 share their first r indices
    x = np.random.default_rng(8).standard_normal(64).astype(np.float32)
    w, C, T = oracle.fixed_point_weights(x, _rho(64, 8))
    a = oracle.draw_indices(C, T, 30, 1, 0, 2)
    b = oracle.draw_indices(C, T, 31, 1, 0, 2)
    assert b[:30] == a
    # different tokens, batch rows and seeds give different streams
    assert oracle.draw_indices(C, T, 30, 1, 0, 3) != a
    assert oracle.draw_indices(C, T, 30, 1, 1, 2) != a
    assert oracle.draw_indices(C, T, 30, 2, 0, 2) != a
