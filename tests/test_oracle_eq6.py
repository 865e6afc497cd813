"""Pin the oracle's Eq. 6 mode (the paper's input-independent probability
p_i = ||W[i]||^2 / ||W||_F^2, one table per weight matrix) against exact rationals,
brute-force enumeration, the closed-form variance (||x||^2 ||W||_F^2 - ||xW||^2) / r,
multi-seed unbiasedness and Lemma 1."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl

W6 = oracle.SAMPLING_WEIGHT


def _exact_sq_norms(W):
    return [sum(Fraction(float(v)) ** 2 for v in row) for row in np.asarray(W, np.float32)]


def test_eq6_table_follows_squared_row_norms():
    rng = np.random.default_rng(3)
    W = (rng.standard_normal((300, 40)) * np.exp(rng.standard_normal((300, 1)))).astype(np.float32)
    w, C, T = oracle.weight_fixed_point(oracle.row_norms(W))
    sq = _exact_sq_norms(W)
    tot = sum(sq)
    for i in range(300):
        p = float(sq[i] / tot)
        # float32 norm, float32 square, 32-bit fixed point: a few float32 ulps
        assert abs(w[i] / T - p) <= 4e-7 * p + 2.0 ** -31, (i, w[i] / T, p)
    assert C[-1] == T == sum(w)


def _power_of_two_rows(d, dout, seed):
    """Rows with 1 or 4 nonzeros of magnitude 2^a: exact norms 2^a or 2^(a+1), so the
    float32 squares and the fixed-point weights are exact and p^ = p."""
    rng = np.random.default_rng(seed)
    W = np.zeros((d, dout), np.float32)
    for i in range(d):
        k = 1 if rng.random() < 0.5 else 4
        cols = rng.choice(dout, k, replace=False)
        W[i, cols] = rng.choice([-1.0, 1.0], k) * 2.0 ** int(rng.integers(-3, 4))
    return W


@pytest.mark.parametrize("d,r", [(3, 1), (3, 2), (4, 2), (4, 3)])
def test_eq6_brute_force_matches_paper_closed_form(d, r):
    dout = 6
    W = _power_of_two_rows(d, dout, 40 + d + r)
    rng = np.random.default_rng(d * 10 + r)
    x = rng.standard_normal(d).astype(np.float32)
    rho = oracle.row_norms(W)
    w, C, T = oracle.weight_fixed_point(rho)
    sq = _exact_sq_norms(W)
    for i in range(d):  # p^ is exactly the paper's p
        assert Fraction(w[i], T) == sq[i] / sum(sq)
    xs = [Fraction(float(v)) for v in x]
    Wq = [[Fraction(float(v)) for v in row] for row in W]
    xW = [sum(xs[i] * Wq[i][c] for i in range(d)) for c in range(dout)]
    E = [Fraction(0)] * dout
    E2 = Fraction(0)
    for tup in itertools.product(range(d), repeat=r):
        p = Fraction(1)
        for s in tup:
            p *= Fraction(w[s], T)
        # H = (1/r) sum_k x_s W_s / p_s, exactly
        H = [sum(xs[s] * Wq[s][c] * Fraction(T, w[s]) for s in tup) / r for c in range(dout)]
        E = [E[c] + p * H[c] for c in range(dout)]
        E2 += p * sum((H[c] - xW[c]) ** 2 for c in range(dout))
        # the oracle's float64 estimate of the same index tuple
        Ho = oracle.estimate_from_indices(x, W, w, T, list(tup), r)
        np.testing.assert_allclose(Ho, [float(h) for h in H], rtol=1e-12, atol=1e-12)
    assert E == xW  # unbiased
    normx2 = sum(v * v for v in xs)
    normW2 = sum(sq)
    assert E2 == (normx2 * normW2 - sum(v * v for v in xW)) / r  # the paper's closed form


def test_eq6_unbiased_over_seeds_and_lemma1():
    rng = np.random.default_rng(9)
    d, dout, r, S = 64, 20, 12, 3000
    x = rng.standard_normal(d).astype(np.float32)
    W = (rng.standard_normal((d, dout)) * np.exp(0.7 * rng.standard_normal((d, 1)))).astype(np.float32)
    rho = oracle.row_norms(W)
    table = oracle.weight_fixed_point(rho)
    w, C, T = table
    exact = x.astype(np.float64) @ W.astype(np.float64)
    Hs = np.stack([oracle.encode_token(x, W, rho, r, seed, 0, 0, sampling=W6, table=table)[0] for seed in range(S)])
    x64, W64 = x.astype(np.float64), W.astype(np.float64)
    var_c = (np.sum((x64[:, None] ** 2) * (W64 ** 2) * T / np.array(w, np.float64)[:, None], axis=0) - exact ** 2) / r
    z = (Hs.mean(axis=0) - exact) / np.sqrt(var_c / S)
    assert np.max(np.abs(z)) < 4.5, z
    # Lemma 1: E||H~ - xW|| <= ||x|| ||W||_F / sqrt(r), and the closed form below the bound
    bound = float(np.linalg.norm(x64) * np.linalg.norm(W64) / np.sqrt(r))
    err = np.linalg.norm(Hs - exact, axis=1)
    assert err.mean() <= bound
    V = oracle.estimator_variance(x, W, w, T, r)
    paper = (float(x64 @ x64) * float(np.sum(W64 ** 2)) - float(exact @ exact)) / r
    assert V == pytest.approx(paper, rel=1e-5)
    assert V <= bound ** 2


def test_eq6_draws_ignore_the_token_and_zero_token_encodes_zero():
    rng = np.random.default_rng(5)
    W = rng.standard_normal((96, 32)).astype(np.float32)
    rho = oracle.row_norms(W)
    x1 = rng.standard_normal(96).astype(np.float32)
    x2 = (3.0 * rng.standard_normal(96)).astype(np.float32)
    _, i1, _ = oracle.encode_token(x1, W, rho, 17, 4, 2, 7, sampling=W6)
    _, i2, _ = oracle.encode_token(x2, W, rho, 17, 4, 2, 7, sampling=W6)
    assert i1 == i2 and len(i1) == 17
    H0, i0, c0 = oracle.encode_token(np.zeros(96, np.float32), W, rho, 17, 4, 2, 7, sampling=W6)
    assert i0 == i1 and np.all(c0 == 0) and np.all(H0 == 0)
    # Eq. 4 mode draws differently for the two tokens and skips the zero token
    _, j1, _ = oracle.encode_token(x1, W, rho, 17, 4, 2, 7)
    _, j2, _ = oracle.encode_token(x2, W, rho, 17, 4, 2, 7)
    assert j1 != j2
    assert oracle.encode_token(np.zeros(96, np.float32), W, rho, 17, 4, 2, 7)[1] == []


def test_eq6_layer_keeps_counts_and_saturated_tokens():
    L = wl.make_layer(2, 24, 48, 2, "f32", data_seed=13, lens=np.array([24, 15]), q_scale=3.0, token_scale_sigma=0.5)
    a = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.3, 5)
    b = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.3, 5, sampling=W6)
    assert np.array_equal(a["r"], b["r"])
    sat = a["r"] == L.d_in
    assert sat.any() and (~sat & (a["r"] > 0)).any()
    np.testing.assert_allclose(b["Htilde"][sat], a["Htilde"][sat], rtol=0, atol=0)
    with pytest.raises(ValueError):
        oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.3, 5, sampling="rows")


def test_non_finite_weights_encode_zero():
    # a row norm whose square overflows float32 leaves no usable distribution
    W = np.ones((8, 4), np.float32)
    W[2] = 3e19
    rho = oracle.row_norms(W)
    assert oracle.weight_fixed_point(rho) is None
    x = np.ones(8, np.float32)
    H, idx, _ = oracle.encode_token(x, W, rho, 3, 0, 0, 0, sampling=W6)
    assert idx == [] and np.all(H == 0)
    assert oracle.fixed_point_weights(np.full(8, 3e38, np.float32), rho) is None
