"""Shared helpers of the GPU parity tests: run a synthetic layer through libmca and
compare its results with the CPU oracle's.

Tolerances (per valid query row i, relative to the row's largest magnitude):
  float32 layers: ||Y_i - Y_i^ref||_inf <= 1e-5 ||Y_i^ref||_inf
  bf16 layers:    ||Y_i - Y_i^ref||_inf <= 2e-2 ||Y_i^ref||_inf (A and H~ enter the P V
                  product in bf16, fp32 accumulation)
  H~ rows (float32 export): 1e-5 in both modes (bf16 inputs are exact in float32 and the
                  gather accumulates in float32)
  column statistic m: a per-key relative bound derived from the inputs and the float32
                  arithmetic of the score pass (``colmax_tolerance``)
Sample counts and sample indices are compared exactly; counts may differ by one only for
tokens whose float64 t^2 lies within that bound of an integer (``ambiguous_tokens``).
"""
from __future__ import annotations

import math

import numpy as np

TOL_Y = {"f32": 1e-5, "bf16": 2e-2}
TOL_H = 1e-5

# ---------------------------------------------------------------- column-max error bound
# The score pass computes, per (batch row, head, query i, key k), in float32:
#   dot~ = q_i . k_k                        MFMA, products of bf16 exact (of float32 rounded),
#                                           float32 accumulation in an unknown order
#   c~_i = M + log2(sum_k exp2(fma(dot~, s32, -M)))   the row normaliser (log2 units),
#                                           s32 = float32(log2(e) / 8)
#   t~   = fma(dot~_ik, s32, -c~_i)         (local window: -(c~_i - log2 |S_i|))
#   m~_k = exp2(max over heads and valid queries of t~)
# against the float64 oracle's m_k = max A = 2^(max t), t = s dot - c, s = log2(e) / 8.
# Error terms (u = 2^-24, gamma_m = m u / (1 - m u), Higham's bound for any summation
# order of m terms):
#   |dot~ - dot| <= e_ik = gamma_65 sum_d |q_d k_d|
#   the scale constant: |s32 - s| |dot|
#   c: c = log2 sum_k 2^(z_k) has gradient p (the row's probabilities) and a Hessian whose
#      quadratic form is at most ln2 |dz|_max^2, so perturbations dz_k of the logits move
#      c by at most sum_k p_k |dz_k| + (ln2 / 2) max_k dz_k^2; the sum L of exp2 terms has
#      relative error <= (u/2) ln2 R (rounding of each fma argument; R the row's logit
#      range) + eps_exp (each exp2) + gamma_{n/16 + 6} (a lane adds its keys in sequence,
#      then four butterfly levels combine 16 lanes), plus, in the streaming kernel, one
#      rescale per visited key tile at most (eps_exp + u each, arguments summing to at
#      most R) and four DPP combination levels; log2 L within 2u max(1, log2 L), where L is
#      the sum under the kernel's reference M (the row's largest logit in its first key
#      tile, or a larger logit of the row once raised), so log2 L is at most the oracle's
#      log2 of the sum under the row max plus (row max - largest logit of tile 0); the
#      add M + log2 L rounds by |c| u / 2
#   t: the fma rounds by |t| u / 2
#   m: exp2 of the maximum: eps_exp; the maximum of perturbed values moves by at most
#      the largest perturbation among the pairs that can be the maximum
# The streaming kernel (rows longer than 8 key tiles) differs in three places: its running
# reference sits up to 16 log2 units below the row max (the exp2 arguments reach R + 16);
# its column statistic starts the MFMA accumulator at d = float32(c~ / s32) and takes
# t~ = s32 max(dot - d): the rounding of d (|c| u / 2) and the accumulation of 64 products
# onto it (gamma_65 |c|, as the products' own term) add to the error of t.
# eps_exp = 2 ulp: v_exp_f32 and v_log_f32 are specified to 1 ulp; a factor of two is kept
# as margin. The mean rule adds the summation of H len probabilities (gamma_{H len});
# the median of perturbed values stays within the largest relative perturbation of all
# the values.
U32 = 2.0 ** -24
EPS_EXP = 2.0 * U32
LOG2E_8 = math.log2(math.e) / 8.0
S32 = float(np.float32(LOG2E_8))


def _gamma(m):
    return m * U32 / (1.0 - m * U32)


def colmax_tolerance(L, importance="max", window=None):
    """Per-key relative bound [B, n] on |m_gpu - m_ref| / m_ref (0 for padded keys)."""
    import oracle

    window = L.window if window is None else window
    B, n, H = L.batch, L.seq, L.heads
    ntiles = (n + 63) // 64
    streaming = ntiles > 8
    ln2 = math.log(2.0)
    ds = abs(S32 - LOG2E_8)
    near_w = 1e-2  # log2 units: pairs this far below a key's maximum cannot become it
    tol = np.zeros((B, n))
    for b in range(B):
        Lb = int(L.lens[b])
        att = oracle.attended(np.arange(Lb), Lb, Lb, window)
        nk = att.sum(axis=1).astype(np.float64)  # keys per query
        ts, Dts = [], []
        for h in range(H):
            cs = slice(64 * h, 64 * h + 64)
            q = L.Q[b, :Lb, cs].astype(np.float64)
            k = L.K[b, :Lb, cs].astype(np.float64)
            dot = q @ k.T
            e = _gamma(65) * (np.abs(q) @ np.abs(k).T)
            z = np.where(att, LOG2E_8 * dot, -np.inf)
            zmax = z.max(axis=1)
            Ls = np.exp2(z - zmax[:, None]).sum(axis=1)
            c = zmax + np.log2(Ls)
            R = zmax - np.where(att, z, np.inf).min(axis=1)
            lgL = np.log2(Ls) + (zmax - z[:, :64].max(axis=1))  # log2 of the sum under tile 0's max
            dL = ln2 * (U32 / 2) * (R + (16.0 if streaming else 0.0)) + EPS_EXP + _gamma(-(-n // 16) + 6)
            if streaming:
                dL = dL + ntiles * (EPS_EXP + U32) + ln2 * (U32 / 2) * R + 4 * (EPS_EXP + 1.5 * U32) \
                     + ln2 * (U32 / 2) * R
            dz = np.where(att, S32 * e + ds * np.abs(dot), 0.0)  # logit perturbations
            P = np.exp2(z - c[:, None])  # the row's probabilities (0 off the pattern)
            dzmax = dz.max(axis=1)
            Ec = (P * dz).sum(axis=1) + (ln2 / 2) * dzmax ** 2 + dL / ln2 * (1 + 1e-6) \
                + 2 * U32 * np.maximum(1.0, lgL) + np.abs(c) * U32 / 2
            t = z - c[:, None]
            if window > 0:  # t = log2(|S_i| A[i, k]) against c~ - log2 |S_i|
                lg = np.log2(nk)
                t = t + lg[:, None]
                Ec = Ec + np.abs(c - lg) * U32 / 2 + 2 * U32 * np.maximum(1.0, lg)
            if streaming:  # the accumulator's start d = c' / s (c' = c, or c - log2 |S_i|)
                cp = np.abs(c - np.log2(nk)) if window > 0 else np.abs(c)
                Ec = Ec + (_gamma(65) * (1 + U32) + U32 / 2) * cp
            Dt = np.where(att, dz + Ec[:, None] + np.abs(np.where(att, t, 0)) * U32 / 2, 0.0)
            ts.append(np.where(att, t, -np.inf))
            Dts.append(Dt)
        # a pair whose t lies more than near_w below a key's maximum cannot become the GPU's
        # maximum when near_w exceeds twice every perturbation; 1e-2 unless the logits are
        # so large that the perturbations reach a quarter of it
        nw = max(near_w, 4.0 * max(float(D.max()) for D in Dts))
        tmax_h = np.stack([t.max(axis=0) for t in ts])
        dnear_h = np.stack([np.where(t >= tm[None, :] - nw, D, 0.0).max(axis=0)
                            for t, D, tm in zip(ts, Dts, tmax_h)])
        dall = np.max(np.stack([D.max(axis=0) for D in Dts]), axis=0)
        if importance == "max":
            T = tmax_h.max(axis=0)
            delta = np.where(tmax_h >= T[None, :] - nw, dnear_h, 0.0).max(axis=0)
            tol[b, :Lb] = np.exp2(delta) * (1 + EPS_EXP) - 1
        else:  # every probability enters the mean or the median
            tol[b, :Lb] = np.exp2(dall) * (1 + EPS_EXP) - 1
            if importance == "mean":
                tol[b, :Lb] += _gamma(H * Lb) + 2 * U32
        tol[b, :Lb] += 1e-12  # the oracle's own float64 rounding
    return tol


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


def ambiguous_tokens(m_ref, lens, alpha, d_in, tol, window=0):
    """Tokens whose count could change when m moves by the relative bound `tol` (a scalar
    or a per-key array like m_ref): the float64 rule's t^2 range
    [t^2 (1-tol)^2, t^2 (1+tol)^2] straddles an integer below d_in. (Local window: m
    carries the per-row factor and t = m / alpha.)"""
    tol = np.broadcast_to(np.asarray(tol, np.float64), m_ref.shape)
    amb = np.zeros(m_ref.shape, bool)
    for b in range(m_ref.shape[0]):
        L = int(lens[b])
        for j in range(L):
            t = (1 if window else L) * float(m_ref[b, j]) / alpha
            lo, hi = (t * (1 - tol[b, j])) ** 2, (t * (1 + tol[b, j])) ** 2

            def rule(tt):
                return d_in if tt >= d_in else max(math.ceil(tt), 1)

            amb[b, j] = rule(lo) != rule(hi)
    return amb


FLT_MIN = 2.0 ** -126  # smallest normal float32


def check_colmax(m_gpu, m_ref, lens, tol):
    """m of every valid key within its bound; padded keys exactly 0. A column maximum
    below the float32 normal range may come out as anything from 0 to FLT_MIN (the
    hardware exp2 flushes subnormal results); its count is 1 either way for any alpha
    above n FLT_MIN. Returns the largest error as a fraction of the bound."""
    valid = np.arange(m_ref.shape[1])[None, :] < np.asarray(lens)[:, None]
    assert np.all(m_gpu[~valid] == 0)
    mg = m_gpu[valid].astype(np.float64)
    mr = m_ref[valid]
    tiny = mr < FLT_MIN
    assert np.all((mg[tiny] >= 0) & (mg[tiny] <= FLT_MIN * (1 + tol[valid][tiny]))), mg[tiny].max()
    rel = np.abs(mg[~tiny] - mr[~tiny]) / mr[~tiny]
    bad = rel > tol[valid][~tiny]
    assert not bad.any(), (rel[bad][:5], tol[valid][~tiny][bad][:5])
    return float((rel / tol[valid][~tiny]).max()) if rel.size else 0.0


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
