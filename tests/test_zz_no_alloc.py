"""mca_attention_forward_noalloc: the forward pass with the library's own scratch array in
place of a caller workspace (for callers that cannot allocate device memory).

GPU: two calls in a row, the second on a smaller layer, each bit-identical to
mca_attention_forward on the same inputs (Y, r, m, H~, sample indices and coefficients).
Host: the size limit and the profiler are rejected before any device work."""
import ctypes

import numpy as np
import pytest

import paper_2201_12854_amd as mca
from paper_2201_12854_amd import binding
from paper_2201_12854_amd import workloads as wl
from mca_testutil import to_device


def _raw_noalloc(desc):
    lib = mca.load_library()
    fake = 1 << 20  # aligned, never dereferenced: every check here runs before device work
    return lib.mca_attention_forward_noalloc(ctypes.byref(desc), fake, fake, fake, fake, fake, fake, fake, None)


def test_noalloc_rejects_oversize_and_profiler():
    big = mca.make_desc(4, 4096, 12, 768, binding.MCA_BF16, 0.4, 0)
    assert mca.workspace_size(big) > binding.MCA_NOALLOC_SCRATCH_BYTES
    assert _raw_noalloc(big) == binding.MCA_ERR_WORKSPACE_TOO_SMALL
    assert "no-allocation entry holds" in mca.load_library().mca_last_error().decode()
    small = mca.make_desc(2, 64, 4, 96, binding.MCA_F32, 0.4, 0)
    small.profiler = 1 << 20
    assert _raw_noalloc(small) == binding.MCA_ERR_INVALID_ARGUMENT
    bad = mca.make_desc(2, 64, 4, 96, binding.MCA_F32, float("nan"), 0)
    assert _raw_noalloc(bad) == binding.MCA_ERR_INVALID_ARGUMENT


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    mca.load_library()
    dev = torch.device("cuda:0")
    layers = [wl.make_layer(8, 128, 768, 12, "bf16", data_seed=61, token_scale_sigma=0.5,
                            lens=np.array([128, 128, 77, 128, 1, 128, 100, 128])),
              wl.make_layer(2, 100, 256, 4, "f32", data_seed=62, lens=np.array([100, 37]), q_scale=2.0,
                            token_scale_sigma=0.5)]
    for L in layers:  # the second call is the smaller one
        print(f"[case] noalloc {L.dtype} B={L.batch} n={L.seq} d_in={L.d_in} H={L.heads}", flush=True)
        desc = mca.make_desc(L.batch, L.seq, L.heads, L.d_in, binding.MCA_BF16 if L.dtype == "bf16" else binding.MCA_F32,
                             0.4, 3)
        assert mca.workspace_size(desc) <= binding.MCA_NOALLOC_SCRATCH_BYTES
        t = to_device(L, dev)
        prep = mca.prepare_weights(t["Wv"])
        kw = dict(heads=L.heads, seq_lens=t["lens"], export=True, export_samples=True)
        a = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, 0.4, 3, **kw)
        b = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, 0.4, 3, noalloc=True, **kw)
        torch.cuda.synchronize()
        r = a.r.cpu().numpy()
        assert ((r > 0) & (r < L.d_in)).any() and (r == 0).any() == (L.lens < L.seq).any()
        for k in ("Y", "r", "colmax", "encoded", "sample_idx", "sample_coef"):
            assert torch.equal(getattr(a, k), getattr(b, k)), k
