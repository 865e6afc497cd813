"""Pin the oracle's row norms (O1), softmax attention (O2) and exact layer (Eq. 1)
against exact arithmetic and an independent library (torch, float64)."""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2201_12854_amd import workloads as wl


def _exact_sqrt_round_f32(S: Fraction) -> np.float32:
    """Correctly rounded float32 of sqrt(S) for a non-negative rational S, by exact
    comparison of squared rounding midpoints."""
    guess = np.float32(np.sqrt(float(S)))
    cands = [guess]
    for _ in range(2):
        cands.append(np.nextafter(cands[-1], np.float32(np.inf)))
    lo = guess
    for _ in range(2):
        lo = np.nextafter(lo, np.float32(0))
        cands.append(lo)
    best = min(cands, key=lambda c: abs(Fraction(float(c)) ** 2 - S))
    # exact: compare against neighbours' midpoints
    up = np.nextafter(best, np.float32(np.inf))
    dn = np.nextafter(best, np.float32(0))
    mid_up = (Fraction(float(best)) + Fraction(float(up))) / 2
    mid_dn = (Fraction(float(best)) + Fraction(float(dn))) / 2
    assert mid_dn ** 2 <= S <= mid_up ** 2
    return best


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_row_norms_correctly_rounded(dtype):
    rng = np.random.default_rng(3)
    W = (0.02 * rng.standard_normal((48, 96))).astype(np.float32)
    W[5] *= 1e-20  # tiny rows
    W[6] = 0.0
    W[7, 3] = 1e30
    if dtype == "bf16":
        W = wl.round_to_bf16(W)
    rho = oracle.row_norms(W)
    assert rho.dtype == np.float32
    mismatches = 0
    for i in range(W.shape[0]):
        S = sum(Fraction(float(v)) ** 2 for v in W[i])
        ref = _exact_sqrt_round_f32(S)
        if rho[i] != ref:
            mismatches += 1
            # only acceptable at a near-tie; then it is the adjacent float32
            assert abs(int(rho[i].view(np.int32)) - int(ref.view(np.int32))) == 1
    assert mismatches == 0
    assert rho[6] == 0.0


def test_row_norms_vs_linalg():
    rng = np.random.default_rng(4)
    W = rng.standard_normal((200, 768)).astype(np.float32)
    rho = oracle.row_norms(W)
    ref = np.linalg.norm(W.astype(np.float64), axis=1)
    assert np.all(np.abs(rho.astype(np.float64) - ref) <= np.spacing(rho.astype(np.float32)))


def test_softmax_vs_torch():
    L = wl.make_layer(2, 40, 64, 2, "f32", data_seed=9, ragged_lens=(7, 40), q_scale=3.0)
    for b in range(2):
        for h in range(2):
            cs = oracle.head_slice(h)
            A = oracle.attention_probs(L.Q[b, :, cs], L.K[b, :, cs], int(L.lens[b]))
            q = torch.from_numpy(L.Q[b, :, cs]).double()
            k = torch.from_numpy(L.K[b, :, cs]).double()
            s = q @ k.T / 8.0
            s[:, int(L.lens[b]):] = float("-inf")
            ref = torch.softmax(s, dim=1).numpy()
            np.testing.assert_allclose(A, ref, rtol=1e-13, atol=1e-300)
            assert np.all(A[:, int(L.lens[b]):] == 0)
            np.testing.assert_allclose(A.sum(axis=1), 1.0, rtol=1e-14)


def test_exact_forward_vs_torch():
    L = wl.make_layer(2, 24, 96, 2, "bf16", data_seed=10, ragged_lens=(5, 24))
    Y = oracle.exact_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads)
    mask = torch.arange(24)[None, :] >= torch.from_numpy(L.lens.astype(np.int64))[:, None]
    for h in range(2):
        cs = oracle.head_slice(h)
        q = torch.from_numpy(L.Q[:, :, cs]).double()
        k = torch.from_numpy(L.K[:, :, cs]).double()
        v = torch.from_numpy(L.X).double() @ torch.from_numpy(L.Wv[:, cs]).double()
        s = q @ k.transpose(1, 2) / 8.0
        s = s.masked_fill(mask[:, None, :], float("-inf"))
        ref = torch.softmax(s, dim=-1) @ v
        np.testing.assert_allclose(Y[:, :, cs], ref.numpy(), rtol=1e-12, atol=1e-14)


def test_column_max_is_over_queries_and_heads():
    # A one-hot attention pattern built through Q: query 3 of head 1 looks only at key 9.
    n, H = 16, 2
    Q = np.zeros((1, n, H * 64), np.float32)
    K = np.zeros((1, n, H * 64), np.float32)
    K[0, 9, 64 + 0] = 1.0
    Q[0, 3, 64 + 0] = 2000.0
    m = oracle.column_max(Q, K, np.array([n]), H)
    assert m[0, 9] == pytest.approx(1.0, abs=1e-12)
    # every other key only receives uniform attention 1/n (head 0) or ~0 from query 3
    others = np.delete(m[0], 9)
    np.testing.assert_allclose(others, 1.0 / n, rtol=1e-12)
