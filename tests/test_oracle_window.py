"""Pin the oracle's local-window mode (Sec. "Longformer": a window of w keys around each
token plus global attention for the first token) and its count rule (Eq. 8 -> Eq. 9 with
the per-row number of attended keys |S_i| in place of n):

* the attention pattern against closed forms (pair counts, symmetry, the global row and
  column) and a set-based construction;
* a window that covers the whole sequence reduces to full attention bit for bit;
* the softmax over each row's attended keys against brute force;
* the rule's defining inequality: sum over j in S_i of A[i, j] / sqrt(r_j) <= alpha for
  every valid row and head (the paper's bound with the factor n replaced by |S_i|), and
  its minimality (one sample fewer breaks it for some row);
* the realised output error against alpha * beta_i * ||W||_F over many seeds.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl


def _pairs_closed_form(L, w):
    """Attended (query, key) pairs among L valid tokens: the band |i - j| <= h, plus the
    first row and column outside the band."""
    h = w // 2
    band = L + 2 * sum(L - d for d in range(1, min(h, L - 1) + 1))
    return band + 2 * max(0, L - 1 - h)


@pytest.mark.parametrize("L,w", [(1, 2), (5, 2), (9, 4), (30, 8), (64, 256), (300, 256), (17, 16)])
def test_attended_pattern_closed_forms(L, w):
    n = L + 3  # padded keys never attended
    M = oracle.attended(np.arange(n), n, L, w)
    V = M[:L, :L]
    assert not M[:, L:].any()
    assert V.sum() == _pairs_closed_form(L, w)
    assert np.array_equal(V, V.T)
    assert V[0].all() and V[:, 0].all()
    S = oracle.keys_attended(L, w)
    h = w // 2
    for i in range(L):
        # set-based construction of row i
        keys = set(range(max(0, i - h), min(L, i + h + 1))) | {0}
        if i == 0:
            keys = set(range(L))
        assert set(np.flatnonzero(V[i]).tolist()) == keys
        assert S[i] == len(keys)
    if L > w + 2:  # interior rows: the band of w + 1 keys and the global key
        assert S[h + 1: L - h].tolist() == [w + 2] * (L - 2 * h - 1)


def test_window_modes_rejected():
    L = wl.make_layer(1, 8, 16, 1, "f32", data_seed=1)
    for w in (-2, 3, 7):
        with pytest.raises(ValueError):
            oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 0, window=w)


def test_window_covering_the_sequence_is_full_attention():
    L = wl.make_layer(2, 40, 48, 2, "f32", data_seed=11, lens=np.array([40, 23]), token_scale_sigma=0.5)
    full = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 3)
    for w in (78, 80, 1000):  # w / 2 >= len - 1
        band = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 3, window=w)
        for b in range(2):
            n = int(L.lens[b])
            # the weighted max is len * max A exactly (scaling by len is monotone)
            np.testing.assert_array_equal(band["m"][b], n * full["m"][b])
        assert np.array_equal(band["r"], full["r"])
        np.testing.assert_array_equal(band["Y"], full["Y"])


def test_banded_softmax_brute_force():
    rng = np.random.default_rng(4)
    n, L, w = 13, 11, 4
    Q = rng.standard_normal((n, 64)).astype(np.float32)
    K = rng.standard_normal((n, 64)).astype(np.float32)
    A = oracle.attention_probs(Q, K, L, w)
    h = w // 2
    for i in range(n):
        keys = [j for j in range(L) if i == 0 or j == 0 or (i - h <= j <= i + h)]
        logits = [sum(float(Q[i, d]) * float(K[j, d]) for d in range(64)) / 8.0 for j in keys]
        mx = max(logits)
        e = [math.exp(v - mx) for v in logits]
        tot = sum(e)
        want = np.zeros(n)
        for j, v in zip(keys, e):
            want[j] = v / tot
        np.testing.assert_allclose(A[i], want, rtol=1e-12, atol=1e-15)
    # the rows of Qbh may start at any position q0
    A5 = oracle.attention_probs(Q[5:8], K, L, w, q0=5)
    np.testing.assert_array_equal(A5, A[5:8])


def _row_sums(Lr, r, window):
    """max over valid rows and heads of sum_{j in S_i, r_j < d_in} A[i, j] / sqrt(r_j)."""
    worst = 0.0
    for b in range(Lr.batch):
        n = int(Lr.lens[b])
        for h in range(Lr.heads):
            cs = oracle.head_slice(h)
            A = oracle.attention_probs(Lr.Q[b, :, cs], Lr.K[b, :, cs], n, window)[:n, :n]
            rb = r[b, :n].astype(np.float64)
            keep = rb < Lr.d_in
            worst = max(worst, float((A[:, keep] / np.sqrt(rb[keep])).sum(axis=1).max()))
    return worst


@pytest.mark.parametrize("alpha", [0.2, 0.4, 1.0])
def test_window_rule_bound_and_minimality(alpha):
    # lengths well past the window
    Lr = wl.make_layer(2, 96, 512, 2, "f32", data_seed=21, lens=np.array([96, 70]), token_scale_sigma=0.5)
    w = 16
    m = oracle.column_max(Lr.Q, Lr.K, Lr.lens, Lr.heads, w)
    r = oracle.sample_counts(m, Lr.lens, alpha, Lr.d_in, w)
    assert (r[r > 0] > 1).mean() > 0.9
    assert _row_sums(Lr, r, w) <= alpha * (1 + 1e-12)
    # minimality: removing one sample from any key with 1 < r_j < d_in breaks the defining
    # inequality sqrt(r_j) >= |S_i| A[i, j] / alpha for some row and head
    for b in range(Lr.batch):
        n = int(Lr.lens[b])
        S = oracle.keys_attended(n, w).astype(np.float64)
        need = np.zeros(n)
        for h in range(Lr.heads):
            cs = oracle.head_slice(h)
            A = oracle.attention_probs(Lr.Q[b, :, cs], Lr.K[b, :, cs], n, w)[:n, :n]
            need = np.maximum(need, ((S[:, None] * A) / alpha).max(axis=0))
        for j in range(n):
            rj = int(r[b, j])
            assert math.sqrt(rj) >= need[j] * (1 - 1e-12) or rj == Lr.d_in
            if 1 < rj < Lr.d_in:
                assert math.sqrt(rj - 1) < need[j] * (1 + 1e-12)


@pytest.mark.parametrize("alpha", [0.3, 0.5])
def test_window_rule_follows_the_global_row(alpha):
    # The first query is zero, so it attends all 80 valid keys uniformly; every other
    # query attends the first key strongly and the rest of its window weakly. The first
    # row then sets most counts, and only its key count |S_0| = 80 (not the window's
    # w + 2 = 18) keeps its error sum within alpha.
    n, w = 80, 16
    Lr = wl.make_layer(1, n, 256, 1, "f32", data_seed=41)
    rng = np.random.default_rng(5)
    u = rng.standard_normal(64)
    u /= np.linalg.norm(u)
    Q = np.tile(4.0 * u, (n, 1)) + 0.05 * rng.standard_normal((n, 64))
    K = 0.05 * rng.standard_normal((n, 64))
    Q[0] = 0.0
    K[0] = 8.0 * u
    Lr.Q = Q[None].astype(np.float32)
    Lr.K = K[None].astype(np.float32)
    m = oracle.column_max(Lr.Q, Lr.K, Lr.lens, Lr.heads, w)
    r = oracle.sample_counts(m, Lr.lens, alpha, Lr.d_in, w)
    assert _row_sums(Lr, r, w) <= alpha * (1 + 1e-12)
    A = oracle.attention_probs(Lr.Q[0, :, :64], Lr.K[0, :, :64], n, w)
    np.testing.assert_allclose(A[0], 1.0 / n, rtol=1e-12)
    short = oracle.sample_counts((w + 2) * A.max(axis=0)[None], Lr.lens, alpha, Lr.d_in, w)
    assert _row_sums(Lr, short, w) > 1.5 * alpha


def test_window_output_error_within_bound():
    # E ||Y~_i - Y_i|| <= alpha beta_i ||W||_F with beta_i the mean ||x_j|| over S_i
    Lr = wl.make_layer(1, 48, 64, 1, "f32", data_seed=31, token_scale_sigma=0.5)
    w, alpha, seeds = 12, 0.8, 40
    Yx = oracle.exact_forward(Lr.Q, Lr.K, Lr.X, Lr.Wv, Lr.lens, Lr.heads, window=w)[0]
    err = np.zeros(48)
    for s in range(seeds):
        Y = oracle.mca_forward(Lr.Q, Lr.K, Lr.X, Lr.Wv, Lr.lens, Lr.heads, alpha, s, window=w)["Y"][0]
        err += np.linalg.norm(Y - Yx, axis=1) / seeds
    M = oracle.attended(np.arange(48), 48, 48, w)
    xn = np.linalg.norm(Lr.X[0].astype(np.float64), axis=1)
    beta = (M * xn[None, :]).sum(axis=1) / M.sum(axis=1)
    bound = alpha * beta * np.linalg.norm(Lr.Wv.astype(np.float64))
    assert (err <= bound).all(), (err / bound).max()
