"""Pin the oracle's two shortcut paths to its full path and to exact arithmetic.

* ``mca_forward(y_rows=R)`` computes only the query rows R of Eq. 5's outer product
  (the GPU tests use it at the 4096-token shape); it must give exactly the rows of
  the full output, including under a local window (where each row's keys depend on
  its position) and for padded query rows.
* ``encode_token(exact_from=k)`` encodes a token exactly once its count reaches k:
  at r = k and r = k + 1 the result is x_j W with no draws (checked against an exact
  rational sum), and at r = k - 1 it is the ordinary estimate with the same draws as
  ``exact_from=0``.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl


@pytest.mark.parametrize("window", [0, 8])
def test_y_rows_equal_full_output_rows(window):
    L = wl.make_layer(2, 37, 24, 4, "f32", data_seed=51, lens=np.array([37, 20]), q_scale=2.0,
                      token_scale_sigma=0.5, window=window)
    full = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 9, window=window)
    # first, last, interior, windowed-interior and padded (row 1 has 20 valid tokens) rows
    rows = [(0, 0), (0, 36), (0, 17), (1, 0), (1, 5), (1, 19), (1, 20), (1, 36)]
    part = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 9, window=window, y_rows=rows)
    assert np.array_equal(part["r"], full["r"])
    assert np.array_equal(part["Htilde"], full["Htilde"])
    want = np.stack([full["Y"][b, i] for b, i in rows])
    np.testing.assert_allclose(part["Y_rows"], want, rtol=1e-13, atol=1e-15)


def _exact_product(x, W):
    """x W with every product and sum in exact rationals, then rounded once."""
    out = []
    for c in range(W.shape[1]):
        acc = Fraction(0)
        for i in range(W.shape[0]):
            acc += Fraction(float(x[i])) * Fraction(float(W[i, c]))
        out.append(float(acc))
    return np.array(out)


@pytest.mark.parametrize("k", [3, 10])
def test_exact_from_switches_at_k(k):
    rng = np.random.default_rng(77 + k)
    d_in, d_out = 16, 6
    x = rng.standard_normal(d_in).astype(np.float32)
    W = rng.standard_normal((d_in, d_out)).astype(np.float32)
    rho = oracle.row_norms(W)
    exact = _exact_product(x, W)
    for r in (k, k + 1):
        H, idx, coef = oracle.encode_token(x, W, rho, r, 5, 0, 3, exact_from=k)
        assert idx == [] and coef.size == 0
        np.testing.assert_allclose(H, exact, rtol=1e-13, atol=1e-13)
    # one below the threshold: the sampled estimate, draw for draw the plain path's
    H, idx, coef = oracle.encode_token(x, W, rho, k - 1, 5, 0, 3, exact_from=k)
    H0, idx0, coef0 = oracle.encode_token(x, W, rho, k - 1, 5, 0, 3)
    assert len(idx) == k - 1 and idx == idx0
    assert np.array_equal(coef, coef0) and np.array_equal(H, H0)
    assert not np.allclose(H, exact)  # a real estimate (16 rows, fewer than 11 draws)
    # the plain path stays sampled at r = k and draws a prefix-extension of r = k - 1
    Hk, idxk, _ = oracle.encode_token(x, W, rho, k, 5, 0, 3)
    assert idxk[:k - 1] == idx0


def test_exact_from_in_the_layer_keeps_counts():
    L = wl.make_layer(1, 30, 40, 4, "f32", data_seed=52, q_scale=3.0, token_scale_sigma=0.5)
    base = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 2, want_samples=True)
    k = int(np.median(base["r"]))
    hyb = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 2, want_samples=True, exact_from=k)
    assert np.array_equal(hyb["r"], base["r"])
    exact_rows = L.X[0].astype(np.float64) @ L.Wv.astype(np.float64)
    for j in range(L.seq):
        r = int(base["r"][0, j])
        if r >= k:
            assert hyb["samples"][(0, j)][0] == []
            np.testing.assert_allclose(hyb["Htilde"][0, j], exact_rows[j], rtol=1e-12, atol=1e-14)
        else:
            assert hyb["samples"][(0, j)][0] == base["samples"][(0, j)][0]
            assert np.array_equal(hyb["Htilde"][0, j], base["Htilde"][0, j])
