"""Pin the oracle's estimator (O7-O9, Eq. 2 and Eq. 5) by brute-force enumeration
in exact rationals, multi-seed unbiasedness, the closed-form variance, Lemma 1
and Theorem 1 (with its Markov tail)."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl


def _token(d, dout, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(d).astype(np.float32)
    W = rng.standard_normal((d, dout)).astype(np.float32)
    return x, W, oracle.row_norms(W)


@pytest.mark.parametrize("d,r", [(2, 1), (3, 2), (4, 3), (4, 1), (3, 3)])
def test_brute_force_expectation_and_variance(d, r):
    x, W, rho = _token(d, 5, 100 + 10 * d + r)
    x[0] *= 3
    w, C, T = oracle.fixed_point_weights(x, rho)
    keep = [i for i in range(d) if w[i] > 0]
    exact_mean = sum(x[i].astype(np.float64) * W[i].astype(np.float64) for i in keep)
    E = np.zeros(5)
    E2 = 0.0
    total_p = Fraction(0)
    outcomes = []
    for tup in itertools.product(range(d), repeat=r):
        p = Fraction(1)
        for s in tup:
            p *= Fraction(w[s], T)
        if p == 0:
            continue
        H = oracle.estimate_from_indices(x, W, w, T, list(tup), r)
        outcomes.append((float(p), H))
        total_p += p
    assert total_p == 1
    for p, H in outcomes:
        E += p * H
    np.testing.assert_allclose(E, exact_mean, rtol=1e-12, atol=1e-12)
    for p, H in outcomes:
        E2 += p * float((H - exact_mean) @ (H - exact_mean))
    V = oracle.estimator_variance(x, W, w, T, r)
    assert E2 == pytest.approx(V, rel=1e-9, abs=1e-12)
    # with every weight positive the estimator is unbiased for the exact product
    if len(keep) == d:
        np.testing.assert_allclose(E, x.astype(np.float64) @ W.astype(np.float64), rtol=1e-12)


def test_closed_form_matches_dkm_textbook_when_unquantised():
    # (Z^2 - ||xW||^2)/r with Z = sum |x_i| ||W_i||: the DKM variance of the optimal p
    x, W, rho = _token(64, 16, 7)
    w, C, T = oracle.fixed_point_weights(x, rho)
    x64, W64 = x.astype(np.float64), W.astype(np.float64)
    Z = float(np.sum(np.abs(x64) * np.linalg.norm(W64, axis=1)))
    ref = (Z * Z - float((x64 @ W64) @ (x64 @ W64))) / 5
    assert oracle.estimator_variance(x, W, w, T, 5) == pytest.approx(ref, rel=1e-6)


def test_multi_seed_unbiased_and_variance():
    d, dout, r, S = 64, 24, 10, 3000
    x, W, rho = _token(d, dout, 11)
    w, C, T = oracle.fixed_point_weights(x, rho)
    exact = x.astype(np.float64) @ W.astype(np.float64)
    Hs = np.stack([oracle.encode_token(x, W, rho, r, seed, 0, 0)[0] for seed in range(S)])
    mean = Hs.mean(axis=0)
    # per-coordinate closed-form variance (1/r)(sum_i x_i^2 W[i,c]^2 T / w_i - (xW)_c^2)
    x64, W64 = x.astype(np.float64), W.astype(np.float64)
    var_c = (np.sum((x64[:, None] ** 2) * (W64 ** 2) * T / np.array(w, dtype=np.float64)[:, None],
                    axis=0) - exact ** 2) / r
    z = (mean - exact) / np.sqrt(var_c / S)
    assert np.max(np.abs(z)) < 4.5, z
    err2 = np.sum((Hs - exact) ** 2, axis=1)
    V = oracle.estimator_variance(x, W, w, T, r)
    se = err2.std(ddof=1) / np.sqrt(S)
    assert abs(err2.mean() - V) < 5 * se, (err2.mean(), V, se)


@pytest.mark.parametrize("r", [1, 4, 16, 64])
def test_lemma1_bound(r):
    x, W, rho = _token(128, 64, 12 + r)
    exact = x.astype(np.float64) @ W.astype(np.float64)
    errs = [np.linalg.norm(oracle.encode_token(x, W, rho, r, s, 0, 1)[0] - exact) for s in range(128)]
    bound = np.linalg.norm(x.astype(np.float64)) * np.linalg.norm(W.astype(np.float64)) / np.sqrt(r)
    assert np.mean(errs) <= bound


def test_one_hot_zero_and_saturated_tokens():
    d, dout = 32, 16
    _, W, rho = _token(d, dout, 13)
    x = np.zeros(d, np.float32)
    for r in (1, 5, 31):
        H, idx, _ = oracle.encode_token(x, W, rho, r, 3, 0, 0)
        assert np.all(H == 0) and idx == []
    x[9] = -2.5
    for r in (1, 5, 31):
        H, idx, _ = oracle.encode_token(x, W, rho, r, 3, 0, 0)
        assert idx == [9] * r
        np.testing.assert_allclose(H, -2.5 * W[9].astype(np.float64), rtol=1e-15)
    x2 = np.random.default_rng(0).standard_normal(d).astype(np.float32)
    H, idx, _ = oracle.encode_token(x2, W, rho, d, 3, 0, 0)
    np.testing.assert_allclose(H, x2.astype(np.float64) @ W.astype(np.float64), rtol=1e-14)


def _layer_errors(L, alpha, seeds):
    Yx = oracle.exact_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads)
    rho = oracle.row_norms(L.Wv)
    errs, errs_h, Ys = [], [], []
    for s in seeds:
        out = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, alpha, s, rho=rho)
        D = out["Y"] - Yx
        errs.append(np.linalg.norm(D, axis=2))
        errs_h.append(np.stack([np.linalg.norm(D[:, :, oracle.head_slice(h)], axis=2)
                                for h in range(L.heads)]))
        Ys.append(out["Y"])
    return np.array(errs), np.array(errs_h), np.array(Ys), Yx, out["r"]


@pytest.mark.parametrize("alpha", [0.2, 0.4, 1.0])
def test_theorem1_bound_and_markov_tail(alpha):
    L = wl.make_layer(2, 32, 64, 2, "f32", data_seed=31, ragged_lens=(12, 32), q_scale=2.0,
                      token_scale_sigma=0.5)
    errs, errs_h, Ys, Yx, r = _layer_errors(L, alpha, range(128))
    WF = np.linalg.norm(L.Wv.astype(np.float64))
    for b in range(2):
        n = int(L.lens[b])
        beta = np.mean(np.linalg.norm(L.X[b, :n].astype(np.float64), axis=1))
        bound = alpha * beta * WF
        e = errs[:, b, :n]
        assert np.all(e.mean(axis=0) <= bound)
        assert np.all(errs_h[:, :, b, :n].mean(axis=0) <= bound)
        for delta in (0.5, 0.2, 0.1):
            assert np.mean(e > bound / delta) <= delta


def test_layer_output_unbiased():
    L = wl.make_layer(1, 16, 32, 1, "f32", data_seed=32)
    S = 1500
    errs, _, Ys, Yx, r = _layer_errors(L, 1.0, range(S))
    assert np.all(r[0] < L.d_in)  # every token sampled, none exact
    mean = Ys.mean(axis=0)
    sd = Ys.std(axis=0, ddof=1) / np.sqrt(S)
    z = (mean - Yx) / np.maximum(sd, 1e-300)
    assert np.max(np.abs(z)) < 5.0
