"""Seeded synthetic inputs for one MCA attention layer.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic. Both the HIP path (through the binding) and the CPU
oracle consume exactly the arrays it returns, so the two sides always see the
same values.

Recipe (the paper's workloads are GLUE / document-classification text run
through trained BERT-family weights; neither the data nor the weights are
available, so BERT-shaped random layers stand in for them):

* ``X ~ N(0, 1)`` of shape ``[B, n, d_in]``; optionally every token row is
  scaled by a log-normal factor (heavy-tailed token norms, hence heavy-tailed
  attention) *before* the projections.
* ``W_q, W_k, W_v ~ N(0, 0.02^2)`` of shape ``[d_in, H * 64]``.
* ``Q = q_scale * X @ W_q`` and ``K = X @ W_k`` in float32, then rounded to
  the layer dtype (bf16 rounding is round-to-nearest-even). ``X`` and ``W_v``
  are rounded the same way. The returned float32 arrays hold the rounded
  values exactly.
* Optional key padding: ``lens[b]`` valid tokens, right padded.
* Optional shared salient keys (long-sequence workload): per (batch, head) a
  random set of keys gets a common direction ``u`` added to its key vector and
  every query gets the matching component, raising those logits by a fixed
  amount over a diffuse background.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

D_HEAD = 64


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    out = rounded.astype(np.uint32).view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.reshape(a.shape)


@dataclass
class Layer:
    """One synthetic attention layer. All float arrays are float32 holding values
    exactly representable in ``dtype``."""

    name: str
    dtype: str  # "f32" or "bf16"
    Q: np.ndarray  # [B, n, H*64]
    K: np.ndarray  # [B, n, H*64]
    X: np.ndarray  # [B, n, d_in]
    Wv: np.ndarray  # [d_in, d_out]; row i = input feature i
    lens: np.ndarray  # [B] int32, 1..n
    heads: int
    alpha: float
    seed: int
    alphas: tuple = ()
    meta: dict = field(default_factory=dict)
    window: int = 0  # 0: full attention; w > 0: local window of w keys, global first token

    @property
    def batch(self) -> int:
        return self.X.shape[0]

    @property
    def seq(self) -> int:
        return self.X.shape[1]

    @property
    def d_in(self) -> int:
        return self.X.shape[2]

    @property
    def d_out(self) -> int:
        return self.Wv.shape[1]

    @property
    def tokens(self) -> int:
        return int(self.lens.sum())

    def subset(self, batches) -> "Layer":
        idx = np.asarray(batches)
        return Layer(self.name + f"[{len(idx)}]", self.dtype, self.Q[idx], self.K[idx],
                     self.X[idx], self.Wv, self.lens[idx], self.heads, self.alpha,
                     self.seed, self.alphas, dict(self.meta), self.window)


def make_layer(batch: int, seq: int, d_in: int, heads: int, dtype: str = "f32", *,
               data_seed: int = 0, alpha: float = 0.4, seed: int = 0, q_scale: float = 1.0,
               token_scale_sigma: float = 0.0, lens: Optional[np.ndarray] = None,
               ragged_lens: Optional[tuple] = None, salient_keys: int = 0,
               salient_bump: float = 6.0, w_std: float = 0.02, name: str = "custom",
               alphas: tuple = (), window: int = 0) -> Layer:
    if dtype not in ("f32", "bf16"):
        raise ValueError(dtype)
    rng = np.random.default_rng(data_seed)
    d_out = heads * D_HEAD
    X = rng.standard_normal((batch, seq, d_in), dtype=np.float32)
    if token_scale_sigma > 0:
        s = np.exp(token_scale_sigma * rng.standard_normal((batch, seq, 1))).astype(np.float32)
        X = X * s
    Wq = (w_std * rng.standard_normal((d_in, d_out))).astype(np.float32)
    Wk = (w_std * rng.standard_normal((d_in, d_out))).astype(np.float32)
    Wv = (w_std * rng.standard_normal((d_in, d_out))).astype(np.float32)
    Q = (np.float32(q_scale) * (X @ Wq)).astype(np.float32)
    K = (X @ Wk).astype(np.float32)
    if salient_keys > 0:
        # Shared salient set per (batch, head): K_j += c*u for j in S and
        # Q_i += (bump*sqrt(64)/c)*u for all i, so u.u = 1 raises the scaled
        # logit of every (i, j in S) pair by about `bump`.
        c = float(np.sqrt(D_HEAD * w_std * w_std * d_in))
        a = salient_bump * np.sqrt(D_HEAD) / c
        for b in range(batch):
            for h in range(heads):
                u = rng.standard_normal(D_HEAD).astype(np.float32)
                u /= np.linalg.norm(u)
                S = rng.choice(seq, size=min(salient_keys, seq), replace=False)
                cols = slice(h * D_HEAD, (h + 1) * D_HEAD)
                K[b, S, cols] += np.float32(c) * u
                Q[b, :, cols] += np.float32(a) * u
    if lens is None:
        if ragged_lens is not None:
            lo, hi = ragged_lens
            lens = rng.integers(lo, hi + 1, size=batch).astype(np.int32)
        else:
            lens = np.full(batch, seq, dtype=np.int32)
    lens = np.asarray(lens, dtype=np.int32)
    if lens.shape != (batch,) or lens.min() < 1 or lens.max() > seq:
        raise ValueError("lens must be [batch] with values in 1..seq")
    if dtype == "bf16":
        Q, K, X, Wv = (round_to_bf16(t) for t in (Q, K, X, Wv))
    return Layer(name, dtype, np.ascontiguousarray(Q), np.ascontiguousarray(K),
                 np.ascontiguousarray(X), np.ascontiguousarray(Wv), lens, heads,
                 float(alpha), int(seed), tuple(alphas) or (float(alpha),), {}, int(window))


# The five BERT-shaped workloads. Error-bound settings: loose 1.0, default 0.4,
# tight 0.2 (the smallest value the paper evaluates).
ALPHA_LOOSE, ALPHA_DEFAULT, ALPHA_TIGHT = 1.0, 0.4, 0.2


def bert_base_f32() -> Layer:
    """BERT-base layer, fp32: batch 1, seq 128, hidden 768, 12 heads."""
    return make_layer(1, 128, 768, 12, "f32", data_seed=1001, name="bert_base_f32_b1_s128",
                      alphas=(ALPHA_DEFAULT, ALPHA_TIGHT, ALPHA_LOOSE))


def bert_base_bf16() -> Layer:
    """BERT-base layer, bf16: batch 32, seq 128, hidden 768, 12 heads, log-normal(0, 0.5)
    token scales."""
    return make_layer(32, 128, 768, 12, "bf16", data_seed=1002, token_scale_sigma=0.5,
                      name="bert_base_bf16_b32_s128",
                      alphas=(ALPHA_DEFAULT, ALPHA_LOOSE, ALPHA_TIGHT))


def bert_large_sharp_bf16() -> Layer:
    """BERT-large layer, bf16: batch 16, seq 512, hidden 1024, 16 heads, queries scaled by 4."""
    return make_layer(16, 512, 1024, 16, "bf16", data_seed=1003, q_scale=4.0,
                      name="bert_large_bf16_b16_s512_q4")


def bert_base_padded_bf16() -> Layer:
    """BERT-base layer, bf16: batch 64, seq 128 padded, lengths uniform in [16, 128]."""
    return make_layer(64, 128, 768, 12, "bf16", data_seed=1004, ragged_lens=(16, 128),
                      name="bert_base_bf16_b64_s128_padded")


def long_seq_bf16() -> Layer:
    """Long-sequence layer, bf16: batch 4, seq 4096, hidden 768, 12 heads, 32 shared salient
    keys per (batch, head) with a +6 logit bump."""
    return make_layer(4, 4096, 768, 12, "bf16", data_seed=1005, salient_keys=32,
                      salient_bump=6.0, name="long_bf16_b4_s4096_salient32")


# Document-classification stand-ins for the local-window (Longformer) experiments: a
# window of 256 keys with a global first token, BERT-base width, documents whose lengths
# are uniform in [mean / 2, 3 mean / 2] around the paper's average lengths of 167 (AAPD),
# 300 (IMDB) and 705 (HND) tokens, padded to the longest possible.
LONGFORMER_WINDOW = 256


def _longformer(batch: int, mean_len: int, data_seed: int, name: str) -> Layer:
    lo, hi = (mean_len + 1) // 2, (3 * mean_len) // 2
    return make_layer(batch, hi, 768, 12, "bf16", data_seed=data_seed, token_scale_sigma=0.5,
                      ragged_lens=(lo, hi), name=name, window=LONGFORMER_WINDOW,
                      alphas=(ALPHA_DEFAULT, ALPHA_LOOSE, ALPHA_TIGHT))


def longformer_aapd_bf16() -> Layer:
    """Local-window layer, bf16: batch 32, lengths around 167 (padded 250), window 256."""
    return _longformer(32, 167, 1006, "longformer_bf16_b32_len167_w256")


def longformer_imdb_bf16() -> Layer:
    """Local-window layer, bf16: batch 16, lengths around 300 (padded 450), window 256."""
    return _longformer(16, 300, 1007, "longformer_bf16_b16_len300_w256")


def longformer_hnd_bf16() -> Layer:
    """Local-window layer, bf16: batch 8, lengths around 705 (padded 1057), window 256."""
    return _longformer(8, 705, 1008, "longformer_bf16_b8_len705_w256")


WORKLOADS = {
    "bert_base_f32": bert_base_f32,
    "bert_base_bf16": bert_base_bf16,
    "bert_large_sharp_bf16": bert_large_sharp_bf16,
    "bert_base_padded_bf16": bert_base_padded_bf16,
    "long_seq_bf16": long_seq_bf16,
    "longformer_aapd_bf16": longformer_aapd_bf16,
    "longformer_imdb_bf16": longformer_imdb_bf16,
    "longformer_hnd_bf16": longformer_hnd_bf16,
}
