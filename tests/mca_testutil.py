"""Shared helpers of the GPU parity tests: run a synthetic layer through libmca and
compare its results with the CPU oracle's.

Tolerances (per valid query row i, relative to the row's largest magnitude):
  float32 layers: ||Y_i - Y_i^ref||_inf <= 1e-5 ||Y_i^ref||_inf
  bf16 layers:    ||Y_i - Y_i^ref||_inf <= 2e-2 ||Y_i^ref||_inf (A and H~ enter the P V
                  product in bf16, fp32 accumulation)
  H~ rows (float32 export): 1e-5 in both modes (bf16 inputs are exact in float32 and the
                  gather accumulates in float32)
  column max m: relative 1e-5 (float32 softmax of float32-accumulated scores)
Sample counts and sample indices are compared exactly.
"""
from __future__ import annotations

import math

import numpy as np

TOL_Y = {"f32": 1e-5, "bf16": 2e-2}
TOL_H = 1e-5
TOL_M = 1e-5


def to_device(L, dev):
    import torch

    dt = torch.float32 if L.dtype == "f32" else torch.bfloat16
    t = {k: torch.from_numpy(getattr(L, k)).to(device=dev).to(dt).contiguous() for k in ("Q", "K", "X", "Wv")}
    t["lens"] = torch.from_numpy(L.lens.astype(np.int32)).to(dev)
    return t


def run_gpu(L, dev, alpha, seed, *, r_in=None, export=True, export_samples=False, tensors=None, prep=None,
            sampling="token", window=None, importance="max", exact_from=0):
    import torch

    import paper_2201_12854_amd as mca

    t = tensors or to_device(L, dev)
    if prep is None:
        prep = mca.prepare_weights(t["Wv"])
    rin = None if r_in is None else torch.from_numpy(np.ascontiguousarray(r_in, dtype=np.int32)).to(dev)
    out = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads,
                                seq_lens=t["lens"], r_in=rin, export=export, export_samples=export_samples,
                                sampling=sampling, window=L.window if window is None else window,
                                importance=importance, exact_from=exact_from)
    torch.cuda.synchronize()
    res = {"Y": out.Y.cpu().numpy(), "r": out.r.cpu().numpy(), "rho": mca.rownorm(prep, L.d_in).cpu().numpy()}
    if export:
        res["m"] = out.colmax.cpu().numpy()
        res["H"] = out.encoded.cpu().numpy()
    if export_samples:
        res["idx"] = out.sample_idx.cpu().numpy()
        res["coef"] = out.sample_coef.cpu().numpy()
    return res


def row_rel_err(Y, Yref, lens):
    """max over valid rows of ||Y_i - Yref_i||_inf / ||Yref_i||_inf."""
    worst = 0.0
    for b in range(len(lens)):
        n = int(lens[b])
        A = np.asarray(Y[b, :n], np.float64)
        R = np.asarray(Yref[b, :n], np.float64)
        den = np.abs(R).max(axis=1)
        num = np.abs(A - R).max(axis=1)
        ok = den > 0
        if np.any(num[~ok] > 0):
            return math.inf
        if ok.any():
            worst = max(worst, float((num[ok] / den[ok]).max()))
    return worst


def ambiguous_tokens(m_ref, lens, alpha, d_in, tol=TOL_M, window=0):
    """Tokens whose count could change when m moves by a relative `tol`: the float64
    rule's t^2 range [t^2 (1-tol)^2, t^2 (1+tol)^2] straddles an integer below d_in.
    (Local window: m carries the per-row factor and t = m / alpha.)"""
    amb = np.zeros(m_ref.shape, bool)
    for b in range(m_ref.shape[0]):
        L = int(lens[b])
        for j in range(L):
            t = (1 if window else L) * float(m_ref[b, j]) / alpha
            lo, hi = (t * (1 - tol)) ** 2, (t * (1 + tol)) ** 2

            def rule(tt):
                return d_in if tt >= d_in else max(math.ceil(tt), 1)

            amb[b, j] = rule(lo) != rule(hi)
    return amb


def check_rule_property(r, m, lens, alpha, d_in, window=0):
    """The counts the GPU reports satisfy Eq. 9 for the m it reports:
    sqrt(r) >= len * m / alpha and r - 1 < (len * m / alpha)^2 unless clamped
    (local window: m / alpha in place of len * m / alpha)."""
    for b in range(len(lens)):
        L = int(lens[b])
        assert np.all(r[b, L:] == 0)
        rb = r[b, :L].astype(np.float64)
        t = (1 if window else L) * m[b, :L].astype(np.float64) / alpha
        assert np.all((rb >= 1) & (rb <= d_in))
        free = rb < d_in
        assert np.all(np.sqrt(rb[free]) >= t[free] * (1 - 1e-12))
        lower = free & (rb > 1)
        assert np.all(rb[lower] - 1 < t[lower] ** 2 * (1 + 1e-12))
        sat = rb == d_in
        assert np.all(t[sat] ** 2 > (d_in - 1) * (1 - 1e-12))


def compare_samples(gpu, ref, L):
    """Exact indices and near-exact coefficients for every sampled token."""
    n_tok = 0
    for (b, j), (idx, coef) in ref["samples"].items():
        r = int(ref["r"][b, j])
        if not idx:
            continue
        n_tok += 1
        got = gpu["idx"][b, j, :r]
        assert np.array_equal(got, np.asarray(idx, np.int32)), (b, j)
        c = gpu["coef"][b, j, :r].astype(np.float64)
        np.testing.assert_allclose(c, coef, rtol=2e-7, atol=0)
    return n_tok
