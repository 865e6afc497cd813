"""Pin the oracle's mean and median importance rules (the more aggressive schemes named
after Eq. 8: the count rule of Eq. 9 with the mean or the median of A[:, j] over valid
queries and heads in place of the max):

* uniform attention: all three statistics equal 1/len, so all three rules give the max
  rule's counts;
* the means of a sequence's keys sum to 1 (every attention row sums to 1);
* median and mean lie between the column's min and max, so their counts never exceed
  the max rule's;
* the median against a brute-force construction (explicit softmax rows, Python's
  statistics.median), for odd and even numbers of values;
* one-hot attention: the median is (nearly) 0 and the mean counts the queries that
  attend a key.
"""
import math
import statistics

import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl

MEAN, MEDIAN, MAX = oracle.IMPORTANCE_MEAN, oracle.IMPORTANCE_MEDIAN, oracle.IMPORTANCE_MAX


def test_uniform_attention_all_rules_agree():
    B, n, H = 2, 40, 3
    Q = np.zeros((B, n, 64 * H), np.float32)
    K = np.random.default_rng(1).standard_normal((B, n, 64 * H)).astype(np.float32)
    lens = np.array([40, 17])
    for rule in (MEAN, MEDIAN):
        m = oracle.column_importance(Q, K, lens, H, rule)
        for b in range(B):
            np.testing.assert_allclose(m[b, :lens[b]], 1.0 / lens[b], rtol=1e-13)
            assert np.all(m[b, lens[b]:] == 0)
        for alpha in (0.2, 0.4, 1.0):
            r = oracle.sample_counts(m, lens, alpha, 64)
            rmax = oracle.sample_counts(oracle.column_max(Q, K, lens, H), lens, alpha, 64)
            assert np.array_equal(r, rmax)
            assert set(r[r > 0].tolist()) == {math.ceil(round(1 / alpha ** 2, 9))}


def test_means_sum_to_one_and_bounds():
    L = wl.make_layer(2, 48, 64, 3, "f32", data_seed=2, lens=np.array([48, 29]), q_scale=3.0,
                      token_scale_sigma=0.5)
    mmax = oracle.column_max(L.Q, L.K, L.lens, L.heads)
    mmean = oracle.column_importance(L.Q, L.K, L.lens, L.heads, MEAN)
    mmed = oracle.column_importance(L.Q, L.K, L.lens, L.heads, MEDIAN)
    for b in range(2):
        n = int(L.lens[b])
        assert abs(mmean[b, :n].sum() - 1.0) < 1e-12
        vals = np.stack([oracle.attention_probs(L.Q[b, :, oracle.head_slice(h)], L.K[b, :, oracle.head_slice(h)], n)
                         [:n, :n] for h in range(L.heads)])
        lo, hi = vals.min(axis=(0, 1)), vals.max(axis=(0, 1))
        assert np.all(mmean[b, :n] <= hi * (1 + 1e-12)) and np.all(mmean[b, :n] >= lo * (1 - 1e-12))
        assert np.all(mmed[b, :n] <= hi * (1 + 1e-12)) and np.all(mmed[b, :n] >= lo * (1 - 1e-12))
        np.testing.assert_allclose(hi, mmax[b, :n], rtol=1e-14)
    for alpha in (0.2, 0.4, 1.0):
        rmax = oracle.sample_counts(mmax, L.lens, alpha, L.d_in)
        for m in (mmean, mmed):
            r = oracle.sample_counts(m, L.lens, alpha, L.d_in)
            assert np.all(r <= rmax) and np.array_equal(r > 0, rmax > 0)
        assert np.any(oracle.sample_counts(mmean, L.lens, alpha, L.d_in) < rmax)


@pytest.mark.parametrize("n,H", [(5, 1), (6, 1), (5, 3), (4, 2)])  # H * n odd and even
def test_median_brute_force(n, H):
    rng = np.random.default_rng(n * 10 + H)
    Q = rng.standard_normal((1, n, 64 * H)).astype(np.float32)
    K = rng.standard_normal((1, n, 64 * H)).astype(np.float32)
    m = oracle.column_importance(Q, K, np.array([n]), H, MEDIAN)
    mm = oracle.column_importance(Q, K, np.array([n]), H, MEAN)
    for j in range(n):
        col = []
        for h in range(H):
            for i in range(n):
                logits = [sum(float(Q[0, i, 64 * h + d]) * float(K[0, k, 64 * h + d]) for d in range(64)) / 8.0
                          for k in range(n)]
                mx = max(logits)
                e = [math.exp(v - mx) for v in logits]
                col.append(e[j] / sum(e))
        assert m[0, j] == pytest.approx(statistics.median(col), rel=1e-12)
        assert mm[0, j] == pytest.approx(sum(col) / len(col), rel=1e-12)


def test_one_hot_attention():
    # query i attends key (i + 1) mod n by a wide margin: every key is the target of one
    # query per head, so its mean is ~1 / n and its median ~0
    n, H = 16, 2
    Q = np.zeros((1, n, 64 * H), np.float32)
    K = np.zeros((1, n, 64 * H), np.float32)
    for h in range(H):
        for i in range(n):
            Q[0, i, 64 * h + i] = 40.0
            K[0, (i + 1) % n, 64 * h + i] = 40.0
    mmean = oracle.column_importance(Q, K, np.array([n]), H, MEAN)
    mmed = oracle.column_importance(Q, K, np.array([n]), H, MEDIAN)
    np.testing.assert_allclose(mmean[0], 1.0 / n, rtol=1e-6)
    assert np.all(mmed[0] < 1e-50)
    assert np.all(oracle.sample_counts(mmed, np.array([n]), 0.2, 64) == 1)
    assert np.all(oracle.column_max(Q, K, np.array([n]), H)[0] > 0.999)


def test_rule_arguments():
    L = wl.make_layer(1, 8, 16, 1, "f32", data_seed=1)
    with pytest.raises(ValueError):
        oracle.column_importance(L.Q, L.K, L.lens, 1, "mode")
    with pytest.raises(ValueError):
        oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, 1, 0.4, 0, window=4, importance=MEAN)
    a = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, 1, 0.4, 0)
    b = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, 1, 0.4, 0, importance=MAX)
    assert np.array_equal(a["r"], b["r"]) and np.array_equal(a["Y"], b["Y"])
