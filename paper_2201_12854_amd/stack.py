"""A stack of MCA attention layers with synthetic weights: how the estimate's error grows
with depth (Sec. "Integration with Compressed Transformers": MCA's error accumulates over
attention layers, so a 6-layer model loses less than a 12-layer one) and how it behaves
with 16-bit weights (Sec. "Performance-Accuracy Trade-off", the quantised models).

Each layer l maps hidden states h [B, n, d] to LayerNorm(h + Y_l) with
Y_l = MCA(Q = h W_q, K = h W_k, X = h, W_v) through libmca; the projections, the residual
and the normalisation are plain torch operations around the library call (model wiring,
not part of the attention path). The exact stack runs the same layers in the paper's
regular mode (every token's count set to d_in, so H~ = X W_v exactly). Weights are drawn
N(0, 0.02^2) per layer from a seed; the layer-norm has no learned scale or shift.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import binding


@dataclass
class StackLayer:
    Wq: object
    Wk: object
    Wv: object
    prepared: object


class SyntheticEncoder:
    """L attention layers of width d with H heads of 64, weights N(0, 0.02^2), in
    float32 or bfloat16, on one device."""

    def __init__(self, layers: int, d: int, heads: int, dtype: str = "bf16", seed: int = 0, device="cuda:0"):
        import torch

        if heads * 64 != d:
            raise ValueError("d must equal heads * 64")
        self.dtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.d, self.heads = d, heads
        self.device = torch.device(device)
        rng = np.random.default_rng(seed)
        self.layers = []
        for _ in range(layers):
            W = [torch.from_numpy((0.02 * rng.standard_normal((d, d))).astype(np.float32)).to(self.device)
                 .to(self.dtype).contiguous() for _ in range(3)]
            self.layers.append(StackLayer(W[0], W[1], W[2], binding.prepare_weights(W[2])))

    def layer_inputs(self, h, l: int):
        """Q = h W_q and K = h W_k of layer l (torch matmul in the stack's dtype)."""
        B, n, d = h.shape
        L = self.layers[l]
        q = (h.reshape(B * n, d) @ L.Wq).reshape(B, n, d).contiguous()
        k = (h.reshape(B * n, d) @ L.Wk).reshape(B, n, d).contiguous()
        return q, k

    def forward(self, x, seq_lens, alpha: float, seed: int = 0, *, exact: bool = False, keep: bool = False,
                sampling: str = "token", window: int = 0):
        """Runs the stack on x [B, n, d] (the stack's dtype). Layer l draws with seed + l.
        ``exact``: regular mode (r_j = d_in for every token). Returns the final hidden
        states, or the list of every layer's output when ``keep``."""
        import torch

        B, n, d = x.shape
        h = x.contiguous()
        r_full = torch.full((B, n), d, dtype=torch.int32, device=x.device) if exact else None
        outs = []
        for l, L in enumerate(self.layers):
            q, k = self.layer_inputs(h, l)
            res = binding.attention_forward(q, k, h, L.Wv, L.prepared, alpha, seed + l, heads=self.heads,
                                            seq_lens=seq_lens, r_in=r_full, sampling=sampling, window=window)
            y = torch.nn.functional.layer_norm(h.float() + res.Y, (d,))
            h = y.to(self.dtype).contiguous()
            if keep:
                outs.append(h)
        return outs if keep else h


def depth_error(enc: SyntheticEncoder, x, seq_lens, alpha: float, seeds, **kw):
    """Mean over seeds of the relative Frobenius error of every layer's output (valid rows
    only) of the MCA stack against the exact stack, and the exact stack's outputs."""
    import torch

    exact = enc.forward(x, seq_lens, alpha, 0, exact=True, keep=True, **kw)
    B, n, d = x.shape
    mask = (torch.arange(n, device=x.device)[None, :] < seq_lens[:, None]).float()[..., None]
    errs = np.zeros(len(enc.layers))
    for s in seeds:
        outs = enc.forward(x, seq_lens, alpha, s, keep=True, **kw)
        for l, (a, e) in enumerate(zip(outs, exact)):
            diff = ((a.float() - e.float()) * mask).norm().item()
            errs[l] += diff / max((e.float() * mask).norm().item(), 1e-30) / len(seeds)
    return errs
