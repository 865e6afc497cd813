#!/usr/bin/env python3
"""Benchmark of the MCA attention forward pass on one MI355X.

Headline workload: the long-sequence layer in bf16 (batch 4, seq 4096, hidden 768, 12
heads of 64; X ~ N(0, 1), W ~ N(0, 0.02^2), Q = X W_q and K = X W_k with 32 shared
salient keys per (batch row, head) raised by a +6 logit bump), alpha = 0.4 (the default
error bound) and seed 0: the largest of the five BERT-shaped layers, 16,384 tokens. One
step = one mca_attention_forward call (scores + row softmax statistics + column max,
count rule, sampler, gather-accumulate, exact encoding of saturated tokens, Y = A H~)
over the whole batch, inputs resident in HBM. The row norms of W_v are computed once per
weight matrix and timed separately (prepare_us).

Prints one JSON line (stdout). Also reported:
  - per-stage kernel times from HIP event pairs that each stage kernel's dispatch stamps
    (on the library's stream), and the roofline of the dominant kernel;
  - the exact layer on the same GPU with torch (X W_v, then fused SDPA or bmm + softmax;
    key-padding masks where the workload has them) and MCA's speed relative to it;
  - the realised reduction of the X W_v work and the paper's attention FLOP ratio (AXW);
  - the other four layers (BERT-base fp32 batch 1, BERT-base bf16 batch 32, BERT-large
    bf16 with sharpened logits, BERT-base padded batch 64), each with its dense baseline;
  - at BERT-base bf16: the loose and tight error bounds, the paper's Eq. 6 probability,
    the mean and median importance rules, the exact layer through the same kernels;
  - error growth over a 12-layer stack; the local-window (Longformer) stand-ins;
  - the CPU oracle timed on this host (one batch row of the headline workload).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MCA attention tokens/s at 1 GPU; % HBM roofline (sampling) / % MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}  # dense MFMA, by input dtype
FP32_VECTOR_PEAK_TFLOPS = 157.3  # published vector fp32 (counts packed FMA)
HEADLINE = "long_seq_bf16"
OTHER_CONFIGS = ("bert_base_f32", "bert_base_bf16", "bert_large_sharp_bf16", "bert_base_padded_bf16")
# kernel that carries each stage at a given padded length (the names rocprofv3 shows)
CSRC = os.path.join(ROOT, "paper_2201_12854_amd", "csrc")
STAGE_SOURCE = {"scores_colmax": "k_attention.hip", "attn_out": "k_attention.hip", "sample": "k_sample.hip",
                "gather": "k_gather.hip", "saturated": "k_gather.hip"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def time_loop(fn, steps, warmup):
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    t0.record()
    for _ in range(steps):
        fn()
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    return t0.elapsed_time(t1) / steps, wall


def upload(L, dev):
    import torch

    dt = torch.float32 if L.dtype == "f32" else torch.bfloat16
    t = {k: torch.from_numpy(getattr(L, k)).to(dev).to(dt).contiguous() for k in ("Q", "K", "X", "Wv")}
    t["lens"] = torch.from_numpy(L.lens.astype(np.int32)).to(dev)
    return t


def kernel_name(stage, L):
    """The kernel a stage launches for this layer (the launch code's choice by padded length)."""
    nt = (L.seq + 63) // 64
    if stage == "scores_colmax":
        return "k_scores_res" if nt <= (4 if L.dtype == "bf16" else 2) else "k_scores_rs" if nt <= 8 else "k_scores_stream"
    if stage == "attn_out":
        return "k_attn_res" if nt <= (4 if L.dtype == "bf16" else 2) else "k_attn_stream"
    return {"sample": "k_sample", "gather": "k_gather", "saturated": "k_saturated_lds"}[stage]


def qk_flops(L):
    """One Q K^T over the attended (query, key) pairs: 2 * 64 * H * sum_b len_b^2 (full attention)."""
    return 2.0 * 64 * L.heads * float(np.sum(L.lens.astype(np.float64) ** 2))


def stage_work(L, r, idx):
    """Algorithmic bytes and flops of every stage for one forward pass.

    Score pass: Q K^T once per sweep over the keys (the streaming pass for rows longer than
    8 key tiles sweeps twice, recomputing the scores once the row normalisers are known;
    the work figure counts every sweep, as the measurement plan counts recomputed passes;
    one_sweep_flops is the single Q K^T). Output pass: Q K^T and A H~. Sampled tokens: s_x d_in + r_j d_out s_W bytes and 2 r_j d_out flops
    (every draw counted; merged duplicates are reported beside it); saturated tokens:
    2 d_in d_out MFMA flops."""
    B, n, d_in, d_out, H = L.batch, L.seq, L.d_in, L.d_out, L.heads
    elem = 4 if L.dtype == "f32" else 2
    lens = L.lens.astype(np.int64)
    qt = 128 if (n + 63) // 64 > 8 else 64
    nparts = H * ((n + qt - 1) // qt)
    sampled = (r > 0) & (r < d_in)
    sat = r == d_in
    distinct = 0
    draws = int(r[sampled].sum())
    for b, j in zip(*np.nonzero(sampled)):
        distinct += len(np.unique(idx[b, j, :r[b, j]]))
    n_sampled, n_sat = int(sampled.sum()), int(sat.sum())
    n_valid = int(lens.sum())
    n_zero = B * n - n_sampled - n_sat
    qk = qk_flops(L)
    streaming = (n + 63) // 64 > 8
    w = {}
    w["scores_colmax"] = dict(bytes=2.0 * B * n * d_out * elem + 4.0 * B * H * n + 4.0 * B * n * nparts,
                              flops=(2 if streaming else 1) * qk, one_sweep_flops=qk)
    w["sample"] = dict(bytes=4.0 * B * n * nparts + n_valid * d_in * elem + 4.0 * d_in + 4.0 * B * n
                       + 8.0 * distinct + n_zero * d_out * elem, flops=0.0)
    gather_bytes = 8.0 * distinct + distinct * d_out * elem + n_sampled * d_out * elem
    sat_bytes = n_sat * (d_in * elem + d_out * elem) + (d_in * d_out * elem if n_sat else 0)
    w["gather"] = dict(bytes=gather_bytes + sat_bytes, flops=2.0 * distinct * d_out + 2.0 * n_sat * d_in * d_out,
                       sampled_flops=2.0 * distinct * d_out,
                       sampled_flops_every_draw=2.0 * draws * d_out,
                       bytes_every_draw=8.0 * distinct + draws * d_out * elem + n_sampled * d_out * elem + sat_bytes,
                       mfma_flops=2.0 * n_sat * d_in * d_out)
    w["attn_out"] = dict(bytes=2.0 * B * n * d_out * elem + B * n * d_out * elem + 4.0 * B * n * d_out
                         + 4.0 * B * H * n, flops=2 * qk)
    w["saturated"] = dict(bytes=sat_bytes, flops=2.0 * n_sat * d_in * d_out)
    stats = dict(sampled_tokens=n_sampled, saturated_tokens=n_sat, draws=draws, distinct_rows=distinct)
    return w, stats


def flop_reduction(L, r):
    """X W_v multiply-adds, dense over sampled (the benchmark spec's figure), and the paper's ratio of
    attention FLOPs A X W (Sec. Experiments: only the attention's FLOPs are counted)."""
    lens = L.lens.astype(np.float64)
    tot = float(np.sum(r))
    xw_dense = float(lens.sum()) * L.d_in
    attn = 2.0 * L.d_out * float(np.sum(lens ** 2))
    return {"vs_dense_xw": xw_dense / tot if tot else None,
            "axw_ratio": (2.0 * xw_dense * L.d_out + attn) / (2.0 * L.d_out * tot + attn),
            "mean_r": float(r[r > 0].mean()), "saturated_frac": float((r == L.d_in).sum() / max(1, (r > 0).sum()))}


def source_sha256(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def measured_traffic(kernel, workload, source):
    """HBM bytes per launch of `kernel` at `workload` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (scaled by the copy-kernel calibration recorded there); None if the
    summary is missing or was taken on a different version of the kernel's source file."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.strip().startswith("- "):
            k, v = line.strip()[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    try:
        if vals.get("source") != source or vals.get("source sha256") != source_sha256(os.path.join(CSRC, source)):
            return None
        f, wr = float(vals["fetch bytes per launch"]), float(vals["write bytes per launch"])
        return {"fetch_bytes": f, "write_bytes": wr, "bytes": f + wr, "source": os.path.relpath(path, ROOT)}
    except (KeyError, ValueError, OSError):
        return None


def copy_calibration(mib):
    """A plain elementwise copy of known size (read mib MiB, write mib MiB): the reference
    for scaling the FETCH_SIZE / WRITE_SIZE counters of a profiled run."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 x elementwise copy of {mib} MiB (read {mib} MiB + write {mib} MiB each)")


def dense_baseline(t, L, steps, warmup):
    """The exact layer (Eq. 1) with torch on the same GPU: V = X W_v, then
    softmax(Q K^T / 8) V with the key-padding mask: fused SDPA, and bmm + softmax where the
    score matrix is small enough to materialise; the faster one is the baseline."""
    import torch
    import torch.nn.functional as F

    B, n, H = L.batch, L.seq, L.heads
    X2 = t["X"].reshape(B * n, L.d_in)
    out = {}
    ragged = not np.all(L.lens == n)
    keep = None
    if ragged:
        keep = (torch.arange(n, device=t["X"].device)[None, :] < t["lens"][:, None])  # [B, n] valid keys
    q4 = t["Q"].view(B, n, H, 64).transpose(1, 2).contiguous()
    k4 = t["K"].view(B, n, H, 64).transpose(1, 2).contiguous()
    mask4 = None if keep is None else keep[:, None, None, :]

    def sdpa_path():
        V = (X2 @ t["Wv"]).view(B, n, H, 64).transpose(1, 2).contiguous()
        return F.scaled_dot_product_attention(q4, k4, V, attn_mask=mask4)

    try:
        out["sdpa_ms"], _ = time_loop(sdpa_path, steps, warmup)
    except Exception as e:  # a backend missing in the installed PyTorch: keep the bmm path
        out["sdpa_error"] = str(e)[:200]
    if B * H * n * n <= (1 << 28):  # at most 1 GB of float32 scores
        q = t["Q"].view(B, n, H, 64).permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
        kT = t["K"].view(B, n, H, 64).permute(0, 2, 3, 1).reshape(B * H, 64, n).contiguous()
        kb = None if keep is None else keep[:, None, None, :].expand(B, H, 1, n).reshape(B * H, 1, n)

        def bmm_path():
            V = (X2 @ t["Wv"]).view(B, n, H, 64).permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
            S = torch.bmm(q, kT).float() * 0.125
            if kb is not None:
                S = S.masked_fill(~kb, float("-inf"))
            P = torch.softmax(S, dim=-1).to(q.dtype)
            return torch.bmm(P, V)

        out["bmm_softmax_ms"], _ = time_loop(bmm_path, steps, warmup)
    out["ms"] = min(v for k, v in out.items() if k.endswith("_ms"))
    out["path"] = "sdpa" if out.get("sdpa_ms") == out["ms"] else "bmm + softmax"
    out["tokens_per_s"] = float(L.tokens) / (out["ms"] * 1e-3)
    return out


def stage_times(mca, t, L, prep, alpha, seed, steps, warmup, **kw):
    """Mean kernel time of every stage (us) from HIP event pairs stamped by each stage
    kernel's dispatch on the library's stream, over `steps` forward passes."""
    import torch

    prof = mca.Profiler()
    plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=t["lens"],
                           profiler=prof, **kw)
    for _ in range(warmup):
        plan.run()
    torch.cuda.synchronize()
    prof.collect()
    for _ in range(steps):
        plan.run()
    torch.cuda.synchronize()
    st = {k: (v[0] / max(v[1], 1)) * 1e3 for k, v in prof.collect().items()}
    prof.close()
    return st


def roofline(L, stage_us, work, workload):
    """The dominant kernel's achieved rate against its peak (algorithmic work per launch over
    the mean launch time)."""
    dom = max(stage_us, key=lambda k: stage_us[k])
    dur = stage_us[dom] * 1e-6
    kname = kernel_name(dom, L)
    if dom == "gather":
        # sampled rows come from a W_v slice held in LDS: bound by LDS reads and float32 FMA
        # issue; the algorithmic FLOPs of the sampled tokens (every draw), not the MFMA work
        ach = work[dom]["sampled_flops_every_draw"] / dur / 1e12
        roof = {"kernel": kname, "bound": "alu", "achieved": ach, "peak": FP32_VECTOR_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": ach / FP32_VECTOR_PEAK_TFLOPS,
                "hbm_view": {"algorithmic_GBps": work[dom]["bytes_every_draw"] / dur / 1e9, "peak": HBM_PEAK_GBS}}
    elif dom == "sample":
        ach = work[dom]["bytes"] / dur / 1e9
        roof = {"kernel": kname, "bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": ach / HBM_PEAK_GBS}
    else:
        peak = MFMA_PEAK_TFLOPS[L.dtype]
        ach = work[dom]["flops"] / dur / 1e12
        roof = {"kernel": kname, "bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                "frac": ach / peak}
        if dom == "scores_colmax":
            sweeps = int(round(work[dom]["flops"] / work[dom]["one_sweep_flops"]))
            roof["work"] = (f"Q K^T once per sweep, {sweeps} sweep(s) per launch (2 x 64 x H x sum len^2 flops each)")
            roof["one_sweep_TFLOPs"] = work[dom]["one_sweep_flops"] / dur / 1e12
        else:
            roof["work"] = "Q K^T and A H~ per launch"
    tr = measured_traffic(kname, workload, STAGE_SOURCE[dom])
    roof["traffic"] = tr["bytes"] if tr else None
    if tr:
        roof["traffic_detail"] = tr
    roof["avg_launch_us"] = stage_us[dom]
    return roof


def run_config(mca, L, dev, alpha, seed, steps, warmup, *, dense=True):
    """MCA on one layer (stage pass first, then the timed forward loop) and its exact baseline."""
    import torch

    t = upload(L, dev)
    prep = mca.prepare_weights(t["Wv"])
    st = stage_times(mca, t, L, prep, alpha, seed, steps, warmup)
    plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=t["lens"])
    ms, wall = time_loop(plan.run, steps, warmup)
    torch.cuda.synchronize()
    r = plan.r.cpu().numpy()
    res = {"workload": L.name, "batch": L.batch, "seq_len": L.seq, "hidden": L.d_in, "heads": L.heads,
           "dtype": L.dtype, "tokens": L.tokens, "ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3),
           "stage_us": st, "flop_reduction": flop_reduction(L, r), "dense_stage_rates": dense_stage_rates(L, st, r)}
    if dense:
        d = dense_baseline(t, L, steps, warmup)
        res["dense_exact"] = d
        res["speedup_vs_dense"] = d["ms"] / ms
    return res, t, prep, plan


def c2_extras(mca, L, t, prep, alpha, seed, steps, warmup):
    """At BERT-base bf16: other error bounds, Eq. 6, mean/median rules, regular mode."""
    import torch

    out = {}
    for a in (1.0, 0.2):
        p = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, a, seed, heads=L.heads, seq_lens=t["lens"])
        ms, _ = time_loop(p.run, steps, warmup)
        out[f"alpha_{a}"] = {"ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3)}
    p = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=t["lens"],
                        sampling="weight")
    ms, _ = time_loop(p.run, steps, warmup)
    out["sampling_eq6"] = {"ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3)}
    for rule in ("mean", "median"):
        p = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=t["lens"],
                            importance=rule)
        ms, _ = time_loop(p.run, steps, warmup)
        torch.cuda.synchronize()
        rr = p.r.cpu().numpy()
        out[f"importance_{rule}"] = {"ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3),
                                     "stage_us": stage_times(mca, t, L, prep, alpha, seed, steps, warmup,
                                                             importance=rule),
                                     **flop_reduction(L, rr)}
        log(f"  {rule} rule: {ms * 1e3:.1f} us/step")
    # the paper's regular mode through the same kernels: every count at d_in, every token
    # encoded exactly on MFMA (the exact layer, computed by this library)
    r_full = torch.full((L.batch, L.seq), L.d_in, dtype=torch.int32, device=t["X"].device)
    p = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=t["lens"],
                        r_in=r_full)
    ms, _ = time_loop(p.run, steps, warmup)
    out["regular_mode"] = {"ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3)}
    return out


def dense_stage_rates(L, st, r=None):
    """MFMA rates of the dense stages against the dtype's dense peak: the score pass (Q K^T
    per sweep: two sweeps beyond 8 key tiles; `one_sweep` counts one), the output pass (Q K^T
    and A H~) and, when it runs, the separate saturated-encoding kernel (2 d_in d_out per
    saturated token)."""
    peak = MFMA_PEAK_TFLOPS[L.dtype]
    qk = qk_flops(L)
    sweeps = 2 if (L.seq + 63) // 64 > 8 else 1
    out = {}
    for stage, flops in (("scores_colmax", sweeps * qk), ("attn_out", 2 * qk)):
        if st.get(stage):
            tf = flops / (st[stage] * 1e-6) / 1e12
            out[stage] = {"TFLOP/s": tf, "mfma_frac": tf / peak}
    if st.get("scores_colmax"):
        out["scores_colmax"]["one_sweep_mfma_frac"] = qk / (st["scores_colmax"] * 1e-6) / 1e12 / peak
    if st.get("saturated") and r is not None:
        tf = 2.0 * float((r == L.d_in).sum()) * L.d_in * L.d_out / (st["saturated"] * 1e-6) / 1e12
        out["saturated"] = {"TFLOP/s": tf, "mfma_frac": tf / peak}
    return out


def dense_window_baseline(t, L, steps, warmup):
    """The exact local-window layer with torch: V = X W_v, then softmax over each query's
    attended keys (window of L.window keys, global first token, key padding) times V."""
    import torch

    B, n, H, h = L.batch, L.seq, L.heads, L.window // 2
    dev = t["X"].device
    i = torch.arange(n, device=dev)
    band = ((i[:, None] - i[None, :]).abs() <= h) | (i[:, None] == 0) | (i[None, :] == 0)
    keep = band[None] & (i[None, None, :] < t["lens"].view(B, 1, 1))  # [B, n, n]
    keep = keep[:, None].expand(B, H, n, n).reshape(B * H, n, n)
    X2 = t["X"].reshape(B * n, L.d_in)
    q = t["Q"].view(B, n, H, 64).permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
    kT = t["K"].view(B, n, H, 64).permute(0, 2, 3, 1).reshape(B * H, 64, n).contiguous()

    def bmm_path():
        V = (X2 @ t["Wv"]).view(B, n, H, 64).permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
        S = torch.bmm(q, kT).float() * 0.125
        P = torch.softmax(S.masked_fill(~keep, float("-inf")), dim=-1).to(q.dtype)
        return torch.bmm(P, V)

    ms, _ = time_loop(bmm_path, steps, warmup)
    return {"ms": ms, "tokens_per_s": float(L.tokens) / (ms * 1e-3), "path": "bmm + masked softmax"}


def window_extras(mca, wl, dev, alpha, seed, steps, warmup):
    """The local-window (Longformer) stand-ins: MCA with the window, the same layer with
    full attention, and the exact windowed layer with torch."""
    import torch

    out = {}
    for name in ("longformer_aapd_bf16", "longformer_imdb_bf16", "longformer_hnd_bf16"):
        L = wl.WORKLOADS[name]()
        t = upload(L, dev)
        prep = mca.prepare_weights(t["Wv"])
        res = {"batch": L.batch, "padded_seq": L.seq, "mean_len": float(L.lens.mean()), "window": L.window,
               "tokens": L.tokens}
        for w in (L.window, 0):
            plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads,
                                   seq_lens=t["lens"], window=w)
            ms, _ = time_loop(plan.run, steps, warmup)
            key = "mca_window" if w else "mca_full_attention"
            res[key] = {"ms_per_step": ms, "tokens_per_s": L.tokens / (ms * 1e-3)}
            if w:
                res[key]["stage_us"] = stage_times(mca, t, L, prep, alpha, seed, steps, warmup, window=w)
                torch.cuda.synchronize()
                r = plan.r.cpu().numpy()
                res[key]["mean_r"] = float(r[r > 0].mean())
                res[key]["saturated_frac"] = float((r == L.d_in).sum() / max(1, (r > 0).sum()))
                res[key]["reduction_vs_dense_xw"] = float(L.tokens * L.d_in) / float(r.sum())
        dense = dense_window_baseline(t, L, steps, warmup)
        res["dense_exact_window"] = dense
        res["speedup_vs_dense"] = dense["ms"] / res["mca_window"]["ms_per_step"]
        log(f"{name}: window {res['mca_window']['ms_per_step'] * 1e3:.1f} us, full attention "
            f"{res['mca_full_attention']['ms_per_step'] * 1e3:.1f} us, dense windowed {dense['ms'] * 1e3:.1f} us")
        out[name] = res
    return out


def depth_extras(dev):
    """Error growth with depth: a 12-layer stack of MCA attention layers (BERT-base width,
    synthetic N(0, 0.02^2) weights, layer-norm after the residual) against the same stack in
    regular mode (exact X W_v), relative Frobenius error of every layer's output averaged
    over 4 seeds, in bfloat16 and float32."""
    import torch

    from paper_2201_12854_amd.stack import SyntheticEncoder, depth_error

    B, n, d, H, layers = 8, 128, 768, 12, 12
    x32 = np.random.default_rng(11).standard_normal((B, n, d)).astype(np.float32)
    lens = torch.full((B,), n, dtype=torch.int32, device=dev)
    out = {"batch": B, "seq": n, "d": d, "heads": H, "layers": layers}
    for dtype in ("bf16", "f32"):
        enc = SyntheticEncoder(layers, d, H, dtype, seed=21, device=dev)
        x = torch.from_numpy(x32).to(dev).to(enc.dtype).contiguous()
        res = {}
        for alpha in (0.2, 0.4, 1.0):
            errs = depth_error(enc, x, lens, alpha, range(1, 5))
            res[str(alpha)] = {"rel_error_by_layer": [float(e) for e in errs], "after_6": float(errs[5]),
                               "after_12": float(errs[11])}
        out[dtype] = res
        log(f"depth ({dtype}): relative error after 1 / 6 / 12 layers at alpha 0.4: "
            + " / ".join(f"{res['0.4']['rel_error_by_layer'][i]:.4f}" for i in (0, 5, 11)))
    return out


def host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = os.cpu_count()
    return {"cpu_model": model, "os_cpu_count": os.cpu_count(), "affinity_cpus": aff,
            "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(L, alpha, seed, seconds):
    """The CPU oracle (fp64 numpy, python loops), as it stands, on whole batch rows of the
    workload, one after another until `seconds` have passed (or all rows are done): O1-O9
    for each row's tokens (row norms, attention, column max, counts, fixed point and draws,
    encoding, Y = A H~). BLAS threads are limited to the CPUs this process may run on (and
    OMP_NUM_THREADS, when set)."""
    import oracle

    info = host_info()
    threads = info["affinity_cpus"] or 1
    if info["OMP_NUM_THREADS"]:
        try:
            threads = min(threads, int(info["OMP_NUM_THREADS"]))
        except ValueError:
            pass
    import contextlib

    try:
        from threadpoolctl import threadpool_limits

        limiter = threadpool_limits(limits=threads)
    except Exception:
        limiter = contextlib.nullcontext()
    rows, tokens = 0, 0
    with limiter:
        t0 = time.perf_counter()
        while rows < L.batch and time.perf_counter() - t0 < seconds:
            # one row as a batch of its own (its draws use batch index 0: other samples, the same work)
            Lb = L.subset([rows])
            oracle.mca_forward(Lb.Q, Lb.K, Lb.X, Lb.Wv, Lb.lens, Lb.heads, alpha, seed)
            rows += 1
            tokens += Lb.tokens
        el = time.perf_counter() - t0
    return {"value": tokens / el, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"the first {rows} of the workload's {L.batch} batch rows ({tokens} of {L.tokens} tokens), each "
                      f"the whole forward of one sequence (O1-O9), run until {seconds:.0f} s had passed: {el:.1f} s; "
                      f"python loops plus numpy BLAS with {threads} thread(s)",
            "host": info}


def issue_probe(rounds=20000):
    """Issue costs on this GPU from libmca_probe.so (independent instruction chains per wave,
    clock stamps per wave, spans taken over each workgroup's waves): cycles per wave64
    instruction per SIMD for v_fma_f32, v_exp_f32, v_max3_f32 and the 16x16x32 bf16 MFMA with
    1, 2 and 4 waves per SIMD, the chip-wide MFMA rate, and how far VALU work and MFMAs
    overlap: in every wave (64 fma or 64 exp with 16 MFMAs per round, 64 exp with 64 fma) and
    split over the two waves of a SIMD. Returns a dict."""
    import ctypes

    import torch

    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2201_12854_amd", "libmca_probe.so")
    if not os.path.exists(path):
        raise SystemExit(f"{path} is missing: build it first (python -m paper_2201_12854_amd.build_lib)")
    torch.cuda.init()
    lib = ctypes.CDLL(path)
    lib.mca_issue_probe.restype = ctypes.c_int
    lib.mca_issue_probe.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_longlong),
                                    ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    names = {0: "fma", 1: "exp", 2: "mfma", 3: "fma+mfma", 4: "fma|mfma", 5: "exp+mfma", 6: "exp|mfma", 7: "max3",
             8: "exp+fma"}

    def run(kind, w):
        cap = 8192
        buf = (ctypes.c_longlong * (4 * cap))()
        nw = ctypes.c_int(0)
        for _ in range(2):  # the first call warms the clocks up
            rc = lib.mca_issue_probe(kind, w, rounds, buf, cap, ctypes.byref(nw))
            if rc != 0:
                raise SystemExit(f"mca_issue_probe({names[kind]}, {w}) failed with {rc}")
        # [workgroup (one per CU)][wave][t0, t1, r0, r1]; spans from the first start to the
        # last end over a workgroup's waves, so that waves which do not run side by side are
        # not taken for overlap
        st = np.frombuffer(buf, dtype=np.int64, count=4 * nw.value).reshape(-1, 4 * w, 4).astype(np.float64)
        span_cyc = st[:, :, 1].max(axis=1) - st[:, :, 0].min(axis=1)
        span_ns = (st[:, :, 3].max(axis=1) - st[:, :, 2].min(axis=1)) * 10.0
        wave_cyc = st[:, :, 1] - st[:, :, 0]
        chip_ns = (st[:, :, 3].max() - st[:, :, 2].min()) * 10.0
        return {"span_cycles": float(np.median(span_cyc)), "clock_ghz": float(np.median(span_cyc / span_ns)),
                "wave_share_of_span": float(np.median(wave_cyc.mean(axis=1) / span_cyc)), "chip_ns": float(chip_ns),
                "waves": nw.value}

    out = {"rounds": rounds, "cycles_per_instr_per_simd": {}, "clock_ghz": {}, "wave_share_of_span": {},
           "mixed_cycles_per_round_per_simd": {}}
    per_round = {0: 64, 1: 64, 2: 16, 7: 64}
    for kind in (0, 1, 7, 2):
        for w in (1, 2, 4):
            r = run(kind, w)
            key = f"{names[kind]}_w{w}"
            out["cycles_per_instr_per_simd"][key] = r["span_cycles"] / (w * rounds * per_round[kind])
            out["clock_ghz"][key] = r["clock_ghz"]
            out["wave_share_of_span"][key] = r["wave_share_of_span"]
            if kind == 2:
                out[f"mfma_bf16_TFLOPs_w{w}"] = r["waves"] * rounds * 16 * 16384 / r["chip_ns"] / 1e3
    # every wave runs 64 VALU and 16 MFMAs per round (w waves per SIMD), or the two halves of
    # a SIMD's two waves do one each: cycles per SIMD for one round of each wave's work
    for kind, ws in ((3, (1, 2, 4)), (5, (1, 2, 4)), (8, (1, 2, 4)), (4, (2,)), (6, (2,))):
        for w in ws:
            r = run(kind, w)
            out["mixed_cycles_per_round_per_simd"][f"{names[kind]}_w{w}"] = r["span_cycles"] / rounds
            out["clock_ghz"][f"{names[kind]}_w{w}"] = r["clock_ghz"]
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--alpha", type=float, default=0.4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="time budget of the CPU oracle baseline")
    ap.add_argument("--no-extras", action="store_true", help="only the headline workload and its dense baseline")
    ap.add_argument("--forward-only", metavar="WORKLOAD", default=None,
                    help="only time the MCA forward of one workload (for profiler runs; no JSON bench line)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run a plain copy of MIB MiB (for scaling rocprofv3 byte counters)")
    ap.add_argument("--issue-probe", action="store_true",
                    help="only measure VALU, exp2 and MFMA issue costs with libmca_probe.so (one JSON object)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the multi-GPU layout is a design "
              "note, not a built path", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2201_12854_amd as mca
    from paper_2201_12854_amd import workloads as wl

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a HIP device")
    dev = torch.device("cuda:0")
    if args.issue_probe:
        print(json.dumps({"issue_probe": issue_probe()}), flush=True)
        return
    if args.forward_only:
        L = wl.WORKLOADS[args.forward_only]()
        t = upload(L, dev)
        prep = mca.prepare_weights(t["Wv"])
        plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                               seq_lens=t["lens"])
        ms, _ = time_loop(plan.run, args.steps, args.warmup)
        log(f"{L.name}: {ms * 1e3:.1f} us/step over {args.steps} steps")
        if args.calibrate_copy:
            copy_calibration(args.calibrate_copy)
        return

    L = wl.WORKLOADS[HEADLINE]()
    log(f"workload {L.name}: B={L.batch} n={L.seq} d={L.d_in} H={L.heads} tokens={L.tokens} alpha={args.alpha}")
    head, t, prep, plan = run_config(mca, L, dev, args.alpha, args.seed, args.steps, args.warmup)
    ms = head["ms_per_step"]
    value = L.tokens / (ms * 1e-3)
    log(f"mca forward: {ms * 1e3:.1f} us/step, {value:.4g} tokens/s; stages "
        + ", ".join(f"{k}={v:.1f}" for k, v in head["stage_us"].items()) + " us")
    log(f"dense exact layer: {head['dense_exact']['ms'] * 1e3:.1f} us/step ({head['dense_exact']['path']})")
    prep_ms, _ = time_loop(lambda: mca.prepare_weights(t["Wv"], prep), 20, 3)

    ex = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                               seq_lens=t["lens"], export_samples=True)
    torch.cuda.synchronize()
    r = ex.r.cpu().numpy()
    idx = ex.sample_idx.cpu().numpy()
    del ex
    work, wstats = stage_work(L, r, idx)
    st = head["stage_us"]
    roof = roofline(L, st, work, L.name)
    stages = {k: {"kernel": kernel_name(k, L), "us": st[k],
                  "GB/s": work[k]["bytes"] / (st[k] * 1e-6) / 1e9 if st[k] else None,
                  "TFLOP/s": work[k]["flops"] / (st[k] * 1e-6) / 1e12 if st[k] else None}
              for k in st}
    record = {"metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
              "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
              "vs_baseline": None, "dtype": "bf16",
              "data": "synthetic: seeded long-sequence layer, random N(0, 0.02^2) weights, 32 shared salient keys "
                      "per (batch row, head) with a +6 logit bump",
              "config": {"workload": L.name, "batch": L.batch, "seq_len": L.seq, "hidden": L.d_in,
                         "heads": L.heads, "d_head": 64, "alpha": args.alpha, "seed": args.seed},
              "roofline": roof, "stages": stages, "dense_exact": head["dense_exact"],
              "speedup_vs_dense": head["speedup_vs_dense"], "dense_stage_rates": head["dense_stage_rates"],
              "prepare_us": prep_ms * 1e3, "flop_reduction": {**head["flop_reduction"], **wstats}}
    del plan, t, prep
    torch.cuda.empty_cache()

    if not args.no_extras:
        configs = {}
        for name in OTHER_CONFIGS:
            Lc = wl.WORKLOADS[name]()
            res, tc, pc, _ = run_config(mca, Lc, dev, args.alpha, args.seed, args.steps, args.warmup)
            log(f"{Lc.name}: {res['ms_per_step'] * 1e3:.1f} us/step, dense {res['dense_exact']['ms'] * 1e3:.1f} us "
                f"({res['speedup_vs_dense']:.2f}x), stages "
                + ", ".join(f"{k}={v:.1f}" for k, v in res["stage_us"].items()))
            if name == "bert_base_bf16":
                res["variants"] = c2_extras(mca, Lc, tc, pc, args.alpha, args.seed, args.steps, args.warmup)
            configs[name] = res
            del tc, pc
        record["other_configs"] = configs
        record["depth"] = depth_extras(dev)
        record["local_window"] = window_extras(mca, wl, dev, args.alpha, args.seed, max(1, args.steps // 4),
                                               max(1, args.warmup // 4))
    if args.calibrate_copy:
        copy_calibration(args.calibrate_copy)
    if not args.no_cpu_baseline:
        record["cpu_baseline"] = cpu_baseline(L, args.alpha, args.seed, args.cpu_seconds)
        log(f"cpu oracle: {record['cpu_baseline']['value']:.4g} tokens/s ({record['cpu_baseline']['sample']})")
    print(json.dumps(record), flush=True)


if __name__ == "__main__":
    main()
