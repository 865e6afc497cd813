#!/usr/bin/env python3
"""Benchmark of the MCA attention forward pass on one MI355X.

Workload: a BERT-base-shaped layer in bf16 (batch 32, seq 128, hidden 768, 12 heads of
64), X ~ N(0, 1) with log-normal(0, 0.5) token scales, W ~ N(0, 0.02^2), Q = X W_q and
K = X W_k, alpha = 0.4 (default error bound) and seed 0. One step = one
mca_attention_forward call (scores + softmax statistics + column max, count rule,
sampler, gather-accumulate, exact encoding of saturated tokens, Y = A H~) over the
whole batch, inputs resident in HBM. The row norms of W_v are computed once per
weight matrix and are timed separately (prepare_us).

Prints one JSON line (stdout). Also reported: per-stage kernel times from HIP events
recorded around each launch on the library's stream, the roofline of the dominant
kernel, the same layer computed exactly (dense) with torch on the same GPU, the
realised FLOP reduction, the loose/tight error-bound settings, the paper's Eq. 6
probability, the mean and median importance rules, the dense stages at the BERT-large and 4096-token shapes, the error growth
over a 12-layer stack, the local-window (Longformer) stand-ins against full attention and
the exact windowed layer, and the CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
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
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16
MFMA_FP32_PEAK_TFLOPS = 157.3
FP32_VECTOR_PEAK_TFLOPS = 157.3  # published vector fp32 (counts packed FMA)


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


def stage_work(L, r, idx, elem):
    """Algorithmic bytes and flops of every stage for one forward pass: per sampled token
    s_x d_in + r_j d_out s_W bytes and 2 r_j d_out flops (every draw counted; merged
    duplicates are also reported), per saturated token 2 d_in d_out MFMA flops."""
    B, n, d_in, d_out, H = L.batch, L.seq, L.d_in, L.d_out, L.heads
    s_in, s_h = elem, elem  # input element size; H~ stored in the input dtype
    lens = L.lens.astype(np.int64)
    nparts = H * ((n + 63) // 64)
    sampled = (r > 0) & (r < d_in)
    sat = r == d_in
    distinct = 0
    draws = int(r[sampled].sum())
    for b, j in zip(*np.nonzero(sampled)):
        distinct += len(np.unique(idx[b, j, :r[b, j]]))
    n_sampled, n_sat = int(sampled.sum()), int(sat.sum())
    n_valid = int(lens.sum())
    n_zero = B * n - n_sampled - n_sat
    qk_flops = 2.0 * H * 64 * float(np.sum(n * lens))  # per pass over all (query, valid key) pairs
    w = {}
    w["scores_colmax"] = dict(bytes=2.0 * B * n * d_out * s_in + 4.0 * B * H * n + 4.0 * B * n * nparts,
                              flops=2 * qk_flops)
    # partials, x rows of valid tokens, rho, r, the lists (8 bytes per distinct row), zero rows
    w["sample"] = dict(bytes=4.0 * B * n * nparts + n_valid * d_in * s_in + 4.0 * d_in + 4.0 * B * n
                       + 8.0 * distinct + n_zero * d_out * s_h, flops=0.0)
    # sampled: lists + one W_v row per distinct sampled row + H~ rows; saturated: x rows, W_v once, H~ rows
    gather_bytes = 8.0 * distinct + distinct * d_out * s_in + n_sampled * d_out * s_h
    sat_bytes = n_sat * (d_in * s_in + d_out * s_h) + (d_in * d_out * s_in if n_sat else 0)
    w["gather"] = dict(bytes=gather_bytes + sat_bytes, flops=2.0 * distinct * d_out + 2.0 * n_sat * d_in * d_out,
                       sampled_bytes=gather_bytes, sampled_flops=2.0 * distinct * d_out,
                       sampled_bytes_every_draw=8.0 * distinct + draws * d_out * s_in + n_sampled * d_out * s_h,
                       sampled_flops_every_draw=2.0 * draws * d_out,
                       bytes_every_draw=8.0 * distinct + draws * d_out * s_in + n_sampled * d_out * s_h + sat_bytes,
                       mfma_flops=2.0 * n_sat * d_in * d_out)
    w["attn_out"] = dict(bytes=2.0 * B * n * d_out * s_in + B * n * d_out * s_h + 4.0 * B * n * d_out
                         + 4.0 * B * H * n, flops=2 * qk_flops)
    # the separate saturated kernel (shapes whose B operand does not fit next to the slice);
    # at this shape the gather encodes the saturated tokens and this stage does not run
    w["saturated"] = dict(bytes=sat_bytes, flops=2.0 * n_sat * d_in * d_out)
    stats = dict(sampled_tokens=n_sampled, saturated_tokens=n_sat, draws=draws, distinct_rows=distinct)
    return w, stats


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_gather_bert_base_bf16_b32_s128_traffic.md")
GATHER_SOURCE = os.path.join(ROOT, "paper_2201_12854_amd", "csrc", "k_gather.hip")


def source_sha256(path):
    import hashlib

    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def measured_traffic():
    """HBM bytes per k_gather launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary (scaled by the copy-kernel calibration recorded there); None if the summary is
    missing or was taken on a different k_gather source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and line.strip().startswith("- "):
            k, v = line.strip()[2:].split(":", 1)
            vals[k.strip()] = v.strip().strip("`")
    try:
        if vals.get("k_gather.hip sha256") != source_sha256(GATHER_SOURCE):
            return None
        return {"fetch_bytes": float(vals["fetch bytes per launch"]), "write_bytes": float(vals["write bytes per launch"]),
                "bytes": float(vals["fetch bytes per launch"]) + float(vals["write bytes per launch"]),
                "source": os.path.relpath(TRAFFIC_FILE, ROOT)}
    except (KeyError, ValueError):
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
    """The exact layer (Eq. 1) with torch on the same GPU: V = X W_v, softmax(Q K^T/8) V."""
    import torch
    import torch.nn.functional as F

    B, n, H = L.batch, L.seq, L.heads
    X2 = t["X"].reshape(B * n, L.d_in)
    out = {}

    def bmm_path():
        V = (X2 @ t["Wv"]).view(B, n, H, 64)
        q = t["Q"].view(B, n, H, 64).permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
        kT = t["K"].view(B, n, H, 64).permute(0, 2, 3, 1).reshape(B * H, 64, n).contiguous()
        v = V.permute(0, 2, 1, 3).reshape(B * H, n, 64).contiguous()
        S = torch.bmm(q, kT).float() * 0.125
        P = torch.softmax(S, dim=-1).to(q.dtype)
        return torch.bmm(P, v)

    ms, _ = time_loop(bmm_path, steps, warmup)
    out["bmm_softmax_ms"] = ms
    if np.all(L.lens == n):
        try:
            from torch.nn.attention import SDPBackend, sdpa_kernel

            q4 = t["Q"].view(B, n, H, 64).transpose(1, 2).contiguous()
            k4 = t["K"].view(B, n, H, 64).transpose(1, 2).contiguous()

            def sdpa_path():
                V = (X2 @ t["Wv"]).view(B, n, H, 64).transpose(1, 2).contiguous()
                with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                    return F.scaled_dot_product_attention(q4, k4, V)

            ms2, _ = time_loop(sdpa_path, steps, warmup)
            out["sdpa_ms"] = ms2
        except Exception as e:  # backend unavailable in the installed PyTorch: keep the bmm path
            out["sdpa_error"] = str(e)[:200]
    out["ms"] = min(v for k, v in out.items() if k.endswith("_ms"))
    out["tokens_per_s"] = float(L.tokens) / (out["ms"] * 1e-3)
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
        t = {k: torch.from_numpy(getattr(L, k)).to(dev).to(torch.bfloat16).contiguous()
             for k in ("Q", "K", "X", "Wv")}
        t["lens"] = torch.from_numpy(L.lens.astype(np.int32)).to(dev)
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
                prof = mca.Profiler()
                pp = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads,
                                     seq_lens=t["lens"], window=w, profiler=prof)
                for _ in range(steps):
                    pp.run()
                torch.cuda.synchronize()
                st = prof.collect()
                prof.close()
                res[key]["stage_us"] = {k: (v[0] / max(v[1], 1)) * 1e3 for k, v in st.items()}
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


def dense_stage_extras(mca, wl, dev, alpha, seed, steps):
    """MFMA rates of the dense stages where they carry the work: BERT-large with sharpened
    logits (every token saturates, so the value encoding is the exact X W_v GEMM) and the
    4096-token sequences. Algorithmic FLOPs over the valid keys and queries: the score pass
    2 H sum(len^2) 64 (one Q K^T), the output pass twice that (Q K^T and A H~), the
    saturated encoding 2 d_in d_out per saturated token; against the bf16 dense peak."""
    import torch

    out = {}
    for name in ("bert_large_sharp_bf16", "long_seq_bf16"):
        L = wl.WORKLOADS[name]()
        t = {k: torch.from_numpy(getattr(L, k)).to(dev).to(torch.bfloat16).contiguous()
             for k in ("Q", "K", "X", "Wv")}
        lens = torch.from_numpy(L.lens.astype(np.int32)).to(dev)
        prep = mca.prepare_weights(t["Wv"])
        prof = mca.Profiler()
        plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, alpha, seed, heads=L.heads, seq_lens=lens,
                               profiler=prof)
        for _ in range(20):  # clocks up before the timed passes
            plan.run()
        torch.cuda.synchronize()
        prof.collect()
        for _ in range(steps):
            plan.run()
        torch.cuda.synchronize()
        st = {k: (v[0] / max(v[1], 1)) * 1e3 for k, v in prof.collect().items()}
        prof.close()
        r = plan.r.cpu().numpy()
        nsat = int((r == L.d_in).sum())
        qk = 2.0 * L.heads * float(np.sum(L.lens.astype(np.float64) ** 2)) * 64
        res = {"batch": L.batch, "seq": L.seq, "d": L.d_in, "heads": L.heads, "stage_us": st,
               "ms_per_step": sum(st.values()) * 1e-3, "saturated_tokens": nsat}

        def rate(flops, us):
            if not us:
                return None
            tf = flops / (us * 1e-6) / 1e12
            return {"TFLOP/s": tf, "mfma_frac": tf / MFMA_BF16_PEAK_TFLOPS}

        res["scores_colmax"] = rate(qk, st["scores_colmax"])
        res["attn_out"] = rate(2 * qk, st["attn_out"])
        if st.get("saturated"):
            res["saturated"] = rate(2.0 * nsat * L.d_in * L.d_out, st["saturated"])
        log(f"{name}: " + ", ".join(f"{k}={v:.1f} us" for k, v in st.items()))
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


def cpu_baseline(L, alpha, seed, seconds):
    """The CPU oracle (fp64 numpy), as it stands, on the same layer."""
    import oracle

    try:
        from threadpoolctl import threadpool_info

        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, alpha, seed)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or el * (reps + 1) / reps > 3 * seconds:
            break
    return {"value": L.tokens * reps / el, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"the whole workload ({L.batch} sequences, {L.tokens} tokens) x {reps} run(s), "
                      f"{el:.1f} s; python loops plus numpy BLAS with {threads} thread(s)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=2000)  # about 0.1 s: clocks settle
    ap.add_argument("--alpha", type=float, default=0.4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="skip dense baseline and other alphas")
    ap.add_argument("--dense-stages-only", type=int, default=0, metavar="STEPS",
                    help="only time the dense stages at the BERT-large and 4096-token shapes over STEPS "
                         "passes each and print their JSON (for counter collection; not the bench line)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run a plain copy of MIB MiB (for scaling rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU layout is a "
              "design note, not a measured path", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2201_12854_amd as mca
    from paper_2201_12854_amd import workloads as wl

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a HIP device")
    dev = torch.device("cuda:0")
    if args.dense_stages_only:
        print(json.dumps(dense_stage_extras(mca, wl, dev, args.alpha, args.seed, args.dense_stages_only)), flush=True)
        return
    L = wl.bert_base_bf16()
    elem = 2
    t = {k: torch.from_numpy(getattr(L, k)).to(dev).to(torch.bfloat16).contiguous() for k in ("Q", "K", "X", "Wv")}
    lens = torch.from_numpy(L.lens.astype(np.int32)).to(dev)
    log(f"workload {L.name}: B={L.batch} n={L.seq} d={L.d_in} H={L.heads} tokens={L.tokens} alpha={args.alpha}")

    prep = mca.prepare_weights(t["Wv"])
    prep_ms, _ = time_loop(lambda: mca.prepare_weights(t["Wv"], prep), 20, 3)

    plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads, seq_lens=lens)
    ms, wall = time_loop(plan.run, args.steps, args.warmup)
    value = L.tokens / (ms * 1e-3)
    log(f"mca forward: {ms * 1e3:.1f} us/step, {value:.4g} tokens/s (wall {wall:.2f} s)")

    # per-stage kernel times: a HIP event pair per stage kernel, stamped by its dispatch at the
    # kernel's start and end (on the library's stream)
    prof = mca.Profiler()
    pplan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                            seq_lens=lens, profiler=prof)
    for _ in range(args.warmup):
        pplan.run()
    torch.cuda.synchronize()
    prof.collect()
    for _ in range(args.steps):
        pplan.run()
    torch.cuda.synchronize()
    st = prof.collect()
    stage_us = {k: (v[0] / max(v[1], 1)) * 1e3 for k, v in st.items()}
    ms_prof, _ = time_loop(pplan.run, args.steps, 0)
    prof.collect()
    log("stage us: " + ", ".join(f"{k}={v:.1f}" for k, v in stage_us.items()))

    ex = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                               seq_lens=lens, export_samples=True)
    torch.cuda.synchronize()
    r = ex.r.cpu().numpy()
    idx = ex.sample_idx.cpu().numpy()
    work, wstats = stage_work(L, r, idx, elem)
    dom = max(stage_us, key=lambda k: stage_us[k])
    dur = stage_us[dom] * 1e-6
    if dom == "gather":
        # Sampled rows are gathered from a W_v slice held in LDS, so the kernel is bound by
        # LDS reads and float32 FMA issue, not HBM. achieved = the algorithmic FLOPs of the
        # sampled tokens (2 r_j d_out per token, every draw counted) per launch over the
        # measured launch duration; the MFMA work on saturated tokens in the same launch is
        # not counted. Executed FLOPs (duplicates merged) are reported beside it.
        ach = work[dom]["sampled_flops_every_draw"] / dur / 1e12
        roof = {"kernel": "k_gather", "bound": "alu", "achieved": ach, "peak": FP32_VECTOR_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": ach / FP32_VECTOR_PEAK_TFLOPS, "traffic": None,
                "executed_TFLOPs": work[dom]["sampled_flops"] / dur / 1e12,
                "hbm_view": {"algorithmic_GBps": work[dom]["bytes_every_draw"] / dur / 1e9, "peak": HBM_PEAK_GBS,
                             "frac": work[dom]["bytes_every_draw"] / dur / 1e9 / HBM_PEAK_GBS,
                             "note": "algorithmic bytes (one W_v row per draw) per launch / duration; W_v is "
                                     "on chip (LDS slices), so this exceeds the HBM roofline"}}
        tr = measured_traffic()
        if tr is not None:
            roof["traffic"] = tr["bytes"]
            roof["traffic_detail"] = tr
    else:
        ach = work[dom]["flops"] / dur / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": ach / MFMA_BF16_PEAK_TFLOPS, "traffic": None}
    roof["avg_launch_us"] = stage_us[dom]
    stages = {k: {"us": stage_us[k], "GB/s": work[k]["bytes"] / (stage_us[k] * 1e-6) / 1e9 if stage_us[k] else None,
                  "TFLOP/s": work[k]["flops"] / (stage_us[k] * 1e-6) / 1e12 if stage_us[k] else None}
              for k in stage_us}
    d_in = L.d_in
    red = {"vs_dense_xw": float(L.tokens * d_in) / float(np.sum(r)),
           "mean_r": float(r[r > 0].mean()), "saturated_frac": float((r == d_in).mean()), **wstats}

    record = {"metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
              "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
              "vs_baseline": None, "dtype": "bf16",
              "data": "synthetic: seeded BERT-base-shaped layer, random N(0, 0.02^2) weights",
              "config": {"workload": L.name, "batch": L.batch, "seq_len": L.seq, "hidden": L.d_in,
                         "heads": L.heads, "d_head": 64, "alpha": args.alpha, "seed": args.seed,
                         "token_scale": "lognormal(0, 0.5)"},
              "roofline": roof, "stages": stages, "ms_per_step_with_stage_events": ms_prof,
              "prepare_us": prep_ms * 1e3, "flop_reduction": red}

    if not args.no_extras:
        dense = dense_baseline(t, L, args.steps, args.warmup)
        record["dense_exact"] = dense
        record["speedup_vs_dense"] = dense["ms"] / ms
        log(f"dense exact layer: {dense['ms'] * 1e3:.1f} us/step")
        other = {}
        for a in (1.0, 0.2):
            p2 = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, a, args.seed, heads=L.heads, seq_lens=lens)
            ms_a, _ = time_loop(p2.run, args.steps, args.warmup)
            other[str(a)] = {"ms_per_step": ms_a, "tokens_per_s": L.tokens / (ms_a * 1e-3)}
        record["other_alphas"] = other
        # the paper's input-independent probability (Eq. 6), same workload and alpha
        p6 = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                             seq_lens=lens, sampling="weight")
        ms6, _ = time_loop(p6.run, args.steps, args.warmup)
        record["sampling_eq6"] = {"ms_per_step": ms6, "tokens_per_s": L.tokens / (ms6 * 1e-3)}
        log(f"mca forward, Eq. 6 sampling: {ms6 * 1e3:.1f} us/step")
        # the mean and median importance rules (same workload and alpha)
        rules = {}
        for rule in ("mean", "median"):
            pr = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                                 seq_lens=lens, importance=rule)
            ms_r, _ = time_loop(pr.run, args.steps, args.warmup)
            torch.cuda.synchronize()
            rr = pr.r.cpu().numpy()
            rules[rule] = {"ms_per_step": ms_r, "tokens_per_s": L.tokens / (ms_r * 1e-3),
                           "mean_r": float(rr[rr > 0].mean()), "saturated_frac": float((rr == L.d_in).mean()),
                           "reduction_vs_dense_xw": float(L.tokens * L.d_in) / float(rr.sum())}
            log(f"mca forward, {rule} rule: {ms_r * 1e3:.1f} us/step, mean r {rules[rule]['mean_r']:.1f}")
        record["importance_rules"] = rules
        # the paper's regular mode through the same kernels: every count at d_in, so every
        # token is encoded exactly on MFMA (the exact layer, computed by this library)
        r_full = torch.full((L.batch, L.seq), L.d_in, dtype=torch.int32, device=dev)
        pe = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                             seq_lens=lens, r_in=r_full)
        ms_e, _ = time_loop(pe.run, args.steps, args.warmup)
        record["regular_mode"] = {"ms_per_step": ms_e, "tokens_per_s": L.tokens / (ms_e * 1e-3)}
        log(f"regular mode (exact, same kernels): {ms_e * 1e3:.1f} us/step")
        # tokens whose count reaches k encoded exactly on MFMA as well (the estimate of the
        # others unchanged): where that pays on this chip
        hyb = {}
        for k in (32, 64, 128, 256):
            ph = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, args.alpha, args.seed, heads=L.heads,
                                 seq_lens=lens, exact_from=k)
            ms_h, _ = time_loop(ph.run, args.steps, args.warmup)
            torch.cuda.synchronize()
            rh = ph.r.cpu().numpy()
            exact = (rh >= k) | (rh >= L.d_in)
            sampled_r = rh[(rh > 0) & ~exact]
            macs = float(exact.sum()) * L.d_in + float(sampled_r.sum())  # X W_v rows: exact d_in, sampled r_j
            hyb[str(k)] = {"ms_per_step": ms_h, "tokens_per_s": L.tokens / (ms_h * 1e-3),
                           "exact_tokens_frac": float(exact.mean()),
                           "reduction_vs_dense_xw": float(L.tokens * L.d_in) / macs}
            log(f"exact from r >= {k}: {ms_h * 1e3:.1f} us/step, {100 * exact.mean():.0f}% of tokens exact")
        record["exact_from"] = hyb
        # dense stages at the MFMA-bound shapes
        record["dense_stages"] = dense_stage_extras(mca, wl, dev, args.alpha, args.seed, 50)
        # error growth over a 12-layer stack
        record["depth"] = depth_extras(dev)
        # local-window attention (Longformer stand-ins), fewer steps
        record["local_window"] = window_extras(mca, wl, dev, args.alpha, args.seed, max(1, args.steps // 4),
                                               max(1, args.warmup // 4))
    if args.calibrate_copy:
        copy_calibration(args.calibrate_copy)
    if not args.no_cpu_baseline:
        record["cpu_baseline"] = cpu_baseline(L, args.alpha, args.seed, args.cpu_seconds)
        log(f"cpu oracle: {record['cpu_baseline']['value']:.4g} tokens/s")
    print(json.dumps(record), flush=True)


if __name__ == "__main__":
    main()
