"""Pin the oracle's count rule (O3-O4, Eq. 9) on cases whose answer the paper fixes."""
import os

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "uniform_attention_counts.txt")


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            a, r = line.split()
            rows.append((float(a), int(r)))
    return rows


@pytest.mark.parametrize("alpha,expected", _golden())
@pytest.mark.parametrize("n,valid", [(128, 128), (128, 64), (64, 16), (32, 1)])
def test_uniform_attention(alpha, expected, n, valid):
    # Q = 0 makes every logit 0: A = 1/valid over the valid keys (exact for powers of two).
    H, d_in = 2, 768
    Q = np.zeros((1, n, H * 64), np.float32)
    K = np.random.default_rng(0).standard_normal((1, n, H * 64)).astype(np.float32)
    lens = np.array([valid])
    m = oracle.column_max(Q, K, lens, H)
    np.testing.assert_array_equal(m[0, :valid], 1.0 / valid)
    r = oracle.sample_counts(m, lens, alpha, d_in)
    assert np.all(r[0, :valid] == expected)
    assert np.all(r[0, valid:] == 0)  # padded keys are not encoded


def test_one_hot_attention_saturates():
    n, H, d_in = 32, 1, 256
    Q = np.zeros((1, n, 64), np.float32)
    K = np.zeros((1, n, 64), np.float32)
    K[0, 5, 0] = 1.0
    Q[0, :, 0] = 4000.0  # every query looks only at key 5
    m = oracle.column_max(Q, K, np.array([n]), H)
    r = oracle.sample_counts(m, np.array([n]), 0.4, d_in)
    assert r[0, 5] == d_in  # (n * 1 / 0.4)^2 = 6400 > d_in: capped, encoded exactly
    assert np.all(r[0, np.arange(n) != 5] == 1)  # A ~ e^-500: t^2 ~ 0 -> at least one sample


def test_counts_monotone_in_alpha_and_scale():
    L = wl.make_layer(2, 64, 128, 2, "f32", data_seed=21, ragged_lens=(10, 64))
    m = oracle.column_max(L.Q, L.K, L.lens, L.heads)
    r2 = oracle.sample_counts(m, L.lens, 0.2, L.d_in)
    r4 = oracle.sample_counts(m, L.lens, 0.4, L.d_in)
    r10 = oracle.sample_counts(m, L.lens, 1.0, L.d_in)
    assert np.all(r2 >= r4) and np.all(r4 >= r10)
    valid = np.arange(64)[None, :] < L.lens[:, None]
    assert np.all(r10[valid] >= 1) and np.all(r2[~valid] == 0)
    # sqrt(r) >= n m / alpha (ceil keeps the bound of Theorem 1), and r - 1 < (n m / alpha)^2
    t = (L.lens[:, None] * m) / 0.4
    ok = valid & (r4 < L.d_in)
    assert np.all(np.sqrt(r4[ok]) >= t[ok] * (1 - 1e-15))
    assert np.all((r4[ok] - 1) < t[ok] ** 2 + 1e-9) or np.all(r4[ok] == 1)


def test_alpha_to_zero_is_regular_mode():
    L = wl.make_layer(1, 16, 64, 1, "f32", data_seed=22)
    out = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, 1, 1e-9, 0, want_exact=True)
    assert np.all(out["r"] == L.d_in)
    np.testing.assert_allclose(out["Y"], out["Yexact"], rtol=0, atol=1e-13)


def test_huge_alpha_gives_one_sample():
    L = wl.make_layer(1, 16, 64, 1, "f32", data_seed=23)
    m = oracle.column_max(L.Q, L.K, L.lens, 1)
    assert np.all(oracle.sample_counts(m, L.lens, 1e12, L.d_in) == 1)


def test_non_finite_column_max_saturates():
    # Eq. 9 with an infinite or undefined m (non-finite scores) asks for unboundedly many
    # samples: the count is capped at d_in (an exactly encoded token), never left at the
    # floor of 1; a zero m gives the floor
    m = np.array([[np.inf, np.nan, 0.0, 1e-300, 1e300]])
    r = oracle.sample_counts(m, np.array([5]), 0.4, 64)
    assert r.tolist() == [[64, 64, 1, 1, 64]]
