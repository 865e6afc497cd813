"""GPU parity of the HIP path (through the C ABI) against the CPU fp64 oracle.

Stage by stage: row norms bit-exact; column max within a per-key bound derived from
the inputs and the float32 arithmetic of the score pass (``colmax_tolerance``); sample
counts equal to the oracle's except where the oracle's own t^2 sits within that bound
of an integer (those may differ by one and must satisfy Eq. 9 for the GPU's m);
with the oracle's counts fed in, sample indices bit-exact, H~ and Y within
tolerance. Sizes span several 64-wide tiles with ragged tails; the five BERT-shaped
workloads run at full size (the long-sequence one is checked on one batch row).
"""
import numpy as np
import pytest

import oracle
from paper_2201_12854_amd import workloads as wl
from mca_testutil import (TOL_H, TOL_Y, ambiguous_tokens, check_colmax, check_rule_property, colmax_tolerance,
                          compare_samples, row_rel_err, run_gpu, to_device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch

    import paper_2201_12854_amd as mca

    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    mca.load_library()
    return torch.device("cuda:0")


def _full_check(L, dev, alpha, seed, *, check_e2e_y=True, sampling="token", importance="max", exact_from=0,
                tol_y=None):
    """Oracle vs GPU on every stage; returns (#ambiguous tokens, #sampled tokens)."""
    tol_y = TOL_Y[L.dtype] if tol_y is None else tol_y
    print(f"[case] {L.name} dtype={L.dtype} B={L.batch} n={L.seq} d_in={L.d_in} H={L.heads} "
          f"alpha={alpha} seed={seed} sampling={sampling} window={L.window} importance={importance} "
          f"exact_from={exact_from}", flush=True)
    ref = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, alpha, seed, want_samples=True, sampling=sampling,
                             window=L.window, importance=importance, exact_from=exact_from)
    t = to_device(L, dev)
    g = run_gpu(L, dev, alpha, seed, tensors=t, sampling=sampling, importance=importance, exact_from=exact_from)
    assert np.array_equal(g["rho"], ref["rho"])
    m_ref = ref["m"]
    tol = colmax_tolerance(L, importance)
    used = check_colmax(g["m"], m_ref, L.lens, tol)
    print(f"[m] max relative error {used:.3f} of the per-key bound (bound {tol.max():.2e})", flush=True)
    check_rule_property(g["r"], g["m"], L.lens, alpha, L.d_in, L.window)
    amb = ambiguous_tokens(m_ref, L.lens, alpha, L.d_in, tol, window=L.window)
    diff = g["r"] != ref["r"]
    assert not np.any(diff & ~amb), np.argwhere(diff & ~amb)[:5]
    assert np.all(np.abs(g["r"] - ref["r"])[amb] <= 1)
    if check_e2e_y and not amb.any():
        assert row_rel_err(g["Y"], ref["Y"], L.lens) <= tol_y
    # counts fixed to the oracle's: indices, coefficients, H~ and Y
    g2 = run_gpu(L, dev, alpha, seed, r_in=ref["r"], export_samples=True, tensors=t, sampling=sampling,
                 importance=importance, exact_from=exact_from)
    assert np.array_equal(g2["r"], ref["r"])
    n_tok = compare_samples(g2, ref, L)
    assert row_rel_err(g2["H"], ref["Htilde"], L.lens) <= TOL_H
    assert row_rel_err(g2["Y"], ref["Y"], L.lens) <= tol_y
    return int(amb.sum()), n_tok


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prepared_weights_bitexact(dev, dtype):
    import torch

    import paper_2201_12854_amd as mca

    for (d_in, d_out, scale) in [(96, 256, 0.02), (768, 768, 0.02), (1024, 1024, 1.0), (7, 1000, 1e-20),
                                 (2048, 2048, 3.0), (45, 512, 1.0)]:
        print(f"[case] prepare {dtype} {d_in}x{d_out}", flush=True)
        W = (scale * np.random.default_rng(d_in).standard_normal((d_in, d_out))).astype(np.float32)
        if dtype == "bf16":
            W = wl.round_to_bf16(W)
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        Wd = torch.from_numpy(W).to(dev).to(tdt)
        prep = mca.prepare_weights(Wd)
        torch.cuda.synchronize()
        assert np.array_equal(mca.rownorm(prep, d_in).cpu().numpy(), oracle.row_norms(W))
        # W_v^T in MFMA fragment order, zero padded: [tile][k step][g][r][e] holds
        # W_v[step * KS + g * E + e][16 * tile + r]
        off = (4 * d_in + 255) // 256 * 256
        pad = (d_in + 127) // 128 * 128
        cpad = (d_out + 15) // 16 * 16
        esz, E = (4, 4) if dtype == "f32" else (2, 8)
        nks = pad // (4 * E)
        raw = prep[off: off + cpad * pad * esz].view(tdt).float().cpu().numpy()
        wt = raw.reshape(cpad // 16, nks, 4, 16, E).transpose(0, 3, 1, 2, 4).reshape(cpad, pad)
        ref = np.zeros((cpad, pad), np.float32)
        ref[:d_out, :d_in] = W.T
        assert np.array_equal(wt, ref)
        # prefix sums of the Eq. 6 weights fp32(rho_i^2) in 32-bit fixed point, uint64
        toff = (off + cpad * pad * esz + 255) // 256 * 256
        table = prep[toff: toff + 8 * d_in].cpu().numpy().view(np.uint64)
        q = oracle.weight_fixed_point(oracle.row_norms(W))
        expect = np.zeros(d_in, np.uint64) if q is None else np.array(q[1], np.uint64)
        assert np.array_equal(table, expect)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("alpha", [0.2, 0.4, 1.0])
def test_small_ragged(dev, dtype, alpha):
    # 2 rows (40 and 23 valid of 40: ragged 64-tiles), d_in 96 (ragged k blocks), 4 heads,
    # sharpened logits so saturated and sampled tokens mix
    L = wl.make_layer(2, 40, 96, 4, dtype, data_seed=5, lens=np.array([40, 23]), q_scale=3.0,
                      token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, alpha, seed=11)
    assert n_tok > 0


@pytest.mark.parametrize("alpha", [0.4, 0.2, 1.0])
def test_bert_base_f32(dev, alpha):
    L = wl.bert_base_f32()
    _full_check(L, dev, alpha, seed=0)


@pytest.mark.parametrize("alpha", [0.4, 1.0, 0.2])
def test_bert_base_bf16(dev, alpha):
    L = wl.bert_base_bf16()
    _full_check(L, dev, alpha, seed=0)


def test_bert_large_sharp_bf16(dev):
    L = wl.bert_large_sharp_bf16()
    amb, n_tok = _full_check(L, dev, 0.4, seed=0)


def test_bert_base_padded_bf16(dev):
    L = wl.bert_base_padded_bf16()
    _full_check(L, dev, 0.4, seed=0)


@pytest.fixture(scope="module")
def long_seq(dev):
    """The 4096-token workload through the GPU once, full batch (m, r and Y exported)."""
    L = wl.long_seq_bf16()
    print(f"[case] {L.name} full batch", flush=True)
    g = run_gpu(L, dev, 0.4, 0, export=True)
    check_rule_property(g["r"], g["m"], L.lens, 0.4, L.d_in)
    return L, g


@pytest.mark.parametrize("row", [0, 1, 2, 3])
def test_long_seq_bf16_counts(long_seq, row):
    # every batch row of the full-batch run: m within its bound, counts equal to the
    # oracle's outside the ambiguity band
    L, g = long_seq
    alpha = 0.4
    Lr = L.subset([row])
    print(f"[case] {L.name} row {row}: oracle column max and counts", flush=True)
    m_ref = oracle.column_max(Lr.Q, Lr.K, Lr.lens, Lr.heads)
    r_ref = oracle.sample_counts(m_ref, Lr.lens, alpha, L.d_in)
    tol = colmax_tolerance(Lr)
    used = check_colmax(g["m"][row:row + 1], m_ref, Lr.lens, tol)
    print(f"[m] row {row}: max relative error {used:.3f} of the per-key bound (bound {tol.max():.2e})", flush=True)
    amb = ambiguous_tokens(m_ref, Lr.lens, alpha, L.d_in, tol)
    diff = g["r"][row] != r_ref[0]
    assert not np.any(diff & ~amb[0]), np.argwhere(diff & ~amb[0])[:5]
    assert np.all(np.abs(g["r"][row] - r_ref[0])[amb[0]] <= 1)


def test_long_seq_bf16_row0(dev, long_seq):
    L, g = long_seq
    alpha, seed = 0.4, 0
    L0 = L.subset([0])
    rows = [(0, i) for i in np.random.default_rng(0).choice(L.seq, 48, replace=False)]
    print(f"[case] {L.name} row 0: oracle forward at 48 query rows", flush=True)
    ref = oracle.mca_forward(L0.Q, L0.K, L0.X, L0.Wv, L0.lens, L0.heads, alpha, seed, y_rows=rows,
                             want_samples=True)
    tol = colmax_tolerance(L0)
    check_colmax(g["m"][:1], ref["m"], L0.lens, tol)
    amb = ambiguous_tokens(ref["m"], L0.lens, alpha, L.d_in, tol)
    diff = g["r"][0] != ref["r"][0]
    assert not np.any(diff & ~amb[0])
    # batch row 0 alone with the oracle's counts: indices, H~ and the sampled Y rows
    print(f"[case] {L.name} row 0 with oracle counts", flush=True)
    g0 = run_gpu(L0, dev, alpha, seed, r_in=ref["r"], export_samples=True)
    compare_samples(g0, ref, L0)
    assert row_rel_err(g0["H"], ref["Htilde"], L0.lens) <= TOL_H
    Ys = np.stack([g0["Y"][0, i] for _, i in rows])[None]
    assert row_rel_err(Ys, ref["Y_rows"][None], np.array([len(rows)])) <= TOL_Y["bf16"]
    # the full-batch run agrees with the single-row run on row 0 where the counts agree
    if not diff.any():
        assert np.array_equal(g["Y"][0], g0["Y"][0])


def test_edge_single_token_rows(dev):
    L = wl.make_layer(3, 1, 64, 4, "f32", data_seed=8)
    for alpha in (0.2, 0.7, 3.0):
        _full_check(L, dev, alpha, seed=5)


def test_edge_len_one_and_full(dev):
    L = wl.make_layer(2, 130, 80, 4, "bf16", data_seed=9, lens=np.array([1, 130]))
    _full_check(L, dev, 0.4, seed=6)


def test_edge_zero_and_one_hot_tokens(dev):
    L = wl.make_layer(1, 70, 128, 4, "f32", data_seed=10)
    L.X[0, 3] = 0.0
    L.X[0, 5] = 0.0
    L.X[0, 5, 17] = -1.25
    L.X[0, 6, :] = 1.0  # equal |x|: p proportional to the row norms
    _full_check(L, dev, 1.0, seed=7)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_wide_dynamic_range(dev, dtype):
    # tokens scaled by 1e+20 and 1e-20 in one layer (the scores are left as drawn): the
    # sampling weights |x| rho span 40 decades across tokens, and each token's fixed point
    # is set by its own largest weight
    L = wl.make_layer(2, 50, 96, 4, dtype, data_seed=17, lens=np.array([50, 31]), q_scale=2.0,
                      token_scale_sigma=0.5)
    L.X[:, 1::3] *= np.float32(1e20)
    L.X[:, 2::3] *= np.float32(1e-20)
    if dtype == "bf16":
        L.X = wl.round_to_bf16(L.X)
    amb, n_tok = _full_check(L, dev, 0.4, seed=8)
    assert n_tok > 0


def test_edge_subnormal_products(dev):
    L = wl.make_layer(1, 20, 64, 4, "f32", data_seed=12)
    L.X[0, 2] *= np.float32(1e-36)  # |x| * rho falls into the float32 subnormal range
    _full_check(L, dev, 1.0, seed=7)


def test_edge_regular_mode_and_one_sample(dev):
    L = wl.make_layer(2, 33, 64, 4, "f32", data_seed=13, lens=np.array([33, 17]))
    ex = oracle.exact_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads)
    g = run_gpu(L, dev, 1e-9, 0)
    assert np.all(g["r"][0] == L.d_in) and np.all(g["r"][1, :17] == L.d_in)
    assert row_rel_err(g["Y"], ex, L.lens) <= 1e-5
    _full_check(L, dev, 1e9, seed=1)  # every token gets one sample


def test_edge_seed_high_bits_and_max_sizes(dev):
    L = wl.make_layer(1, 24, 2048, 32, "bf16", data_seed=14, w_std=0.01)
    _full_check(L, dev, 0.6, seed=(1 << 63) + 12345)


def test_edge_d_in_one(dev):
    L = wl.make_layer(2, 9, 1, 4, "f32", data_seed=15, lens=np.array([9, 4]))
    _full_check(L, dev, 0.4, seed=3)


def test_determinism(dev):
    L = wl.bert_base_bf16()
    t = to_device(L, dev)
    a = run_gpu(L, dev, 0.4, 0, tensors=t, export_samples=True)
    b = run_gpu(L, dev, 0.4, 0, tensors=t, export_samples=True)
    for k in ("Y", "r", "m", "H", "idx", "coef"):
        assert np.array_equal(a[k], b[k]), k
    c = run_gpu(L, dev, 0.4, 1, tensors=t)
    assert not np.array_equal(a["Y"], c["Y"])  # another seed, other samples


def test_gpu_estimator_unbiased(dev):
    # the mean of H~ over many seeds converges to x_j W_v (closed-form per-coordinate variance)
    L = wl.make_layer(1, 16, 64, 4, "f32", data_seed=16)
    r = np.full((1, 16), 12, np.int32)
    t = to_device(L, dev)
    S = 400
    Hs = np.stack([run_gpu(L, dev, 1.0, s, r_in=r, tensors=t)["H"][0] for s in range(S)])
    exact = L.X[0].astype(np.float64) @ L.Wv.astype(np.float64)
    rho = oracle.row_norms(L.Wv)
    W64 = L.Wv.astype(np.float64)
    for j in range(16):
        w, C, T = oracle.fixed_point_weights(L.X[0, j], rho)
        x = L.X[0, j].astype(np.float64)
        var_c = (np.sum(x[:, None] ** 2 * W64 ** 2 * T / np.array(w, np.float64)[:, None], axis=0)
                 - exact[j] ** 2) / 12
        z = (Hs[:, j].mean(axis=0) - exact[j]) / np.sqrt(var_c / S)
        assert np.max(np.abs(z)) < 5.5, (j, np.max(np.abs(z)))


# ---------------------------------------------------------------- Eq. 6 sampling mode
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("alpha", [0.2, 0.4, 1.0])
def test_eq6_small_ragged(dev, dtype, alpha):
    L = wl.make_layer(2, 40, 96, 4, dtype, data_seed=5, lens=np.array([40, 23]), q_scale=3.0,
                      token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, alpha, seed=11, sampling="weight")
    assert n_tok > 0


def test_eq6_bert_base_bf16(dev):
    L = wl.bert_base_bf16()
    _full_check(L, dev, 0.4, L.seed, sampling="weight")


def test_eq6_zero_and_one_hot_tokens(dev):
    # under Eq. 6 a zero token still draws (coefficients 0, H~ = 0); a one-hot token keeps one row
    L = wl.make_layer(1, 32, 64, 4, "f32", data_seed=21, q_scale=1.0)
    L.X[0, 3] = 0.0
    L.X[0, 5] = 0.0
    L.X[0, 5, 17] = 2.5
    r_in = np.full((1, 32), 9, np.int64)
    print("[case] eq6 zero / one-hot tokens", flush=True)
    ref = oracle.mca_forward(L.Q, L.K, L.X, L.Wv, L.lens, L.heads, 0.4, 3, r_override=r_in, want_samples=True,
                             sampling="weight")
    g = run_gpu(L, dev, 0.4, 3, r_in=r_in, export_samples=True, sampling="weight")
    compare_samples(g, ref, L)
    assert np.all(g["H"][0, 3] == 0) and np.all(g["coef"][0, 3, :9] == 0)
    assert len(ref["samples"][(0, 3)][0]) == 9
    assert row_rel_err(g["H"], ref["Htilde"], L.lens) <= TOL_H


def test_eq6_draws_do_not_depend_on_x(dev):
    L1 = wl.make_layer(1, 32, 64, 4, "bf16", data_seed=23)
    L2 = wl.make_layer(1, 32, 64, 4, "bf16", data_seed=23)
    L2.X = wl.round_to_bf16(L2.X[:, ::-1, :].copy() * 1.5)
    r_in = np.full((1, 32), 13, np.int64)
    print("[case] eq6 draws independent of x", flush=True)
    g1 = run_gpu(L1, dev, 0.4, 7, r_in=r_in, export_samples=True, sampling="weight")
    g2 = run_gpu(L2, dev, 0.4, 7, r_in=r_in, export_samples=True, sampling="weight")
    assert np.array_equal(g1["idx"][..., :13], g2["idx"][..., :13])
    t1 = run_gpu(L1, dev, 0.4, 7, r_in=r_in, export_samples=True)
    t2 = run_gpu(L2, dev, 0.4, 7, r_in=r_in, export_samples=True)
    assert not np.array_equal(t1["idx"][..., :13], t2["idx"][..., :13])


def test_sampled_d_in_1024_bf16(dev):
    # d_in 1024: 8 tokens per sampler block, the gather's global-memory MFMA operand path
    L = wl.make_layer(2, 64, 1024, 16, "bf16", data_seed=31, q_scale=3.0, token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, 0.4, seed=41)
    assert n_tok > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_saturated_kernel_d_in_1000(dev, dtype):
    # d_in 1000 (above 768, a multiple of 8 but not of 32): the saturated tokens go to the
    # separate staged MFMA kernel, whose last k step re-reads each row's final chunk against
    # the zero padding of the prepared W_v^T. Its blocks of 128 tokens (bf16; 64 for float32)
    # hold 31 to 76 saturated tokens of ragged rows, so some use one row of waves and some
    # both, with partial tiles
    L = wl.make_layer(3, 150, 1000, 8, dtype, data_seed=52, lens=np.array([150, 97, 130]), q_scale=4.0,
                      token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, 0.25, seed=7)
    assert n_tok > 0


def test_bf16_width_not_multiple_of_8(dev):
    # d_in 100: element-wise x loads in the gather, partial lane runs in the sampler
    L = wl.make_layer(2, 48, 100, 4, "bf16", data_seed=32, lens=np.array([48, 29]), q_scale=3.0,
                      token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, 0.4, seed=42)
    assert n_tok > 0


def test_eq6_max_sizes(dev):
    # d_in 2048, 32 heads: 8 tokens per block around a 2048-row shared table
    L = wl.make_layer(1, 24, 2048, 32, "bf16", data_seed=14, w_std=0.01)
    _full_check(L, dev, 0.6, seed=(1 << 63) + 777, sampling="weight")


def test_eq6_d_in_1024(dev):
    L = wl.make_layer(2, 64, 1024, 16, "bf16", data_seed=33, q_scale=3.0, token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, 0.4, seed=43, sampling="weight")
    assert n_tok > 0


# ------------------------------------------------------------------ local-window attention
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("window", [2, 16, 78])
def test_window_small_ragged(dev, dtype, window):
    # resident kernels (n = 40 <= 256); window 78 covers the whole sequence
    L = wl.make_layer(2, 40, 96, 4, dtype, data_seed=5, lens=np.array([40, 23]), q_scale=3.0,
                      token_scale_sigma=0.5, window=window)
    amb, n_tok = _full_check(L, dev, 0.4, seed=11)
    assert n_tok > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("window,lens", [(64, (400, 333)), (128, (300, 1)), (256, (399, 130))])
def test_window_streaming_ragged(dev, dtype, window, lens):
    # streaming kernels (n = 400 > 256): query tiles visit tile 0 and the tiles their
    # window reaches; rows of length 1 and rows shorter than the window
    L = wl.make_layer(2, 400, 128, 4, dtype, data_seed=6, lens=np.array(lens), q_scale=2.0,
                      token_scale_sigma=0.5, window=window)
    amb, n_tok = _full_check(L, dev, 0.4, seed=3)
    assert n_tok > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,lens,window", [(300, (300, 181), 0), (600, (600, 531), 0), (600, (600, 77), 128),
                                           (449, (449, 449), 0), (577, (577, 320), 0)])
def test_score_pass_variants_ragged(dev, dtype, n, lens, window):
    # n = 300: the one-sweep score pass that keeps every score in registers (up to 8 key
    # tiles); n = 600: the two-sweep streaming score pass (its online row sum and its
    # column max), with full attention and with a window; ragged rows. n = 449 and 577 end
    # with a key tile that holds one valid row, so the tile loads' range check covers all
    # but the first row of that tile (one-sweep and streaming kernels, both passes)
    L = wl.make_layer(2, n, 128, 4, dtype, data_seed=9, lens=np.array(lens), q_scale=2.5,
                      token_scale_sigma=0.5, window=window)
    amb, n_tok = _full_check(L, dev, 0.4, seed=5)
    assert n_tok > 0


@pytest.mark.parametrize("n,window,lens", [(520, 126, (520, 301)), (777, 256, (700, 777)), (640, 190, (640, 65)),
                                            (900, 512, (899, 450))])
def test_window_streaming_shapes(dev, n, window, lens):
    # streaming passes under windows of several widths: key tiles that every query of a
    # wave attends whole skip their mask, the others are masked; ragged rows move the
    # boundary of "whole" (keys below len) and windows wider than 2 x 64 + 32 leave
    # interior tiles on both sides of the diagonal
    L = wl.make_layer(2, n, 96, 4, "bf16", data_seed=31 + n, lens=np.array(lens), q_scale=2.0,
                      token_scale_sigma=0.5, window=window)
    amb, n_tok = _full_check(L, dev, 0.4, seed=11)
    assert n_tok > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_streaming_passes_widest_rows(dev, dtype):
    # 32 heads (d_out 2048, the widest row the library takes) with rows of 600 keys, one of
    # them ragged: both streaming passes load their key and H~ tiles through descriptors
    # whose row pitch is the largest allowed
    L = wl.make_layer(1, 600, 128, 32, dtype, data_seed=21, lens=np.array([537]), q_scale=2.0,
                      token_scale_sigma=0.5)
    amb, n_tok = _full_check(L, dev, 0.4, seed=9)
    assert n_tok > 0


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("bump", [20.0, 30.0, 40.0, 100.0])
@pytest.mark.parametrize("n", [700, 480, 250])
def test_score_pass_raised_reference(dev, dtype, bump, n):
    # a few shared keys with a large logit bump (20 is about 29 in log2 units) at random
    # places in the rows: a query that meets one after its first tile adds terms far above
    # its reference logit (its largest logit in tile 0). At bump 100 (144 log2 units) some
    # of them pass the 127 log2 units a float32 term can take, so a score pass that sums
    # under tile 0's largest logit must notice the overflow: the streaming kernel (n = 700)
    # redoes its first sweep with a raised reference and rescaled sums, the one-sweep kernel
    # that streams up to 8 key tiles (n = 480) sums its registers again under the row max.
    # The kernel with every key tile resident (n = 250) takes the row max first. The large
    # logits also stretch the float32 error of the column max (the row normaliser reaches
    # |c| near 60 at bump 40), which the per-key bound must still cover.
    lens = np.array([n, (n * 4) // 5 - 5])
    L = wl.make_layer(2, n, 128, 4, dtype, data_seed=12, lens=lens, salient_keys=6,
                      salient_bump=bump, token_scale_sigma=0.5)
    q = L.Q.astype(np.float64).reshape(2, n, 4, 64)
    k = L.K.astype(np.float64).reshape(2, n, 4, 64)
    lg = np.einsum("bqhd,bkhd->bhqk", q, k) * (np.log2(np.e) / 8)  # logits, log2 units
    if bump == 100.0:  # the input does reach the overflow: some query's logit lies > 127 above tile 0's
        assert np.any(lg.max(axis=3) - lg[..., :64].max(axis=3) > 127)
    # the float32 logit and its row normaliser each carry a rounding error of about
    # |logit| 2^-24, which moves a probability by ln 2 times that: above ~70 log2 units
    # this, not the 1e-5 of the float32 path, bounds the output's relative error
    tol_y = max(TOL_Y[dtype], 4 * np.log(2) * 2.0 ** -24 * np.abs(lg).max())
    amb, n_tok = _full_check(L, dev, 0.4, seed=4, tol_y=tol_y)
    assert n_tok > 0


@pytest.mark.parametrize("rule", ["mean", "median"])
def test_importance_rules_long_rows(dev, rule):
    # mean and median rules through the two-sweep streaming score pass (n = 600)
    L = wl.make_layer(2, 600, 128, 4, "bf16", data_seed=10, lens=np.array([600, 413]), q_scale=2.0,
                      token_scale_sigma=0.5)
    _full_check(L, dev, 0.1, seed=2, importance=rule)


@pytest.mark.parametrize("name", ["longformer_aapd_bf16", "longformer_imdb_bf16", "longformer_hnd_bf16"])
def test_longformer_workloads(dev, name):
    # the document-classification stand-ins at full width, on two batch rows each
    L = wl.WORKLOADS[name]().subset([0, 1])
    for alpha in (0.4, 0.2):
        _full_check(L, dev, alpha, seed=0)


def test_window_eq6(dev):
    L = wl.make_layer(2, 300, 128, 4, "bf16", data_seed=8, lens=np.array([300, 201]), token_scale_sigma=0.5,
                      window=64)
    _full_check(L, dev, 0.4, seed=1, sampling="weight")


# ------------------------------------------------------------------ stacked layers
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stack_layers_match_oracle(dev, dtype):
    # every layer of a 3-layer stack with synthetic weights, on the hidden states the stack
    # itself produced (post layer-norm), against the oracle
    import torch

    from paper_2201_12854_amd.stack import SyntheticEncoder

    enc = SyntheticEncoder(3, 256, 4, dtype, seed=7)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rng = np.random.default_rng(3)
    x = torch.from_numpy(rng.standard_normal((2, 48, 256)).astype(np.float32)).to(dev).to(tdt).contiguous()
    lens_np = np.array([48, 30], np.int32)
    lens = torch.from_numpy(lens_np).to(dev)
    outs = enc.forward(x, lens, 0.4, 5, keep=True)
    torch.cuda.synchronize()
    for l in range(3):
        h = x if l == 0 else outs[l - 1]
        q, k = enc.layer_inputs(h, l)
        arr = [t.float().cpu().numpy() for t in (q, k, h, enc.layers[l].Wv)]
        L = wl.Layer(f"stack_layer{l}", dtype, *arr, lens_np, 4, 0.4, 5 + l)
        _full_check(L, dev, 0.4, seed=5 + l)
    # the exact stack (every count at d_in) equals the regular-mode layers: no samples drawn
    ex = enc.forward(x, lens, 0.4, 5, exact=True)
    assert torch.isfinite(ex.float()).all()


# ------------------------------------------------------------------ mean / median rules
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rule", ["mean", "median"])
def test_importance_rules_small_ragged(dev, dtype, rule):
    # resident kernels; 4 heads x lengths 40 and 23 (H len even and odd for the median)
    L = wl.make_layer(2, 40, 96, 4, dtype, data_seed=5, lens=np.array([40, 23]), q_scale=3.0,
                      token_scale_sigma=0.5)
    for alpha in (0.2, 0.05):
        _full_check(L, dev, alpha, seed=11, importance=rule)


@pytest.mark.parametrize("rule", ["mean", "median"])
def test_importance_rules_streaming(dev, rule):
    L = wl.make_layer(2, 300, 128, 4, "bf16", data_seed=6, lens=np.array([300, 181]), q_scale=2.0,
                      token_scale_sigma=0.5)
    _full_check(L, dev, 0.1, seed=3, importance=rule)


@pytest.mark.parametrize("rule", ["mean", "median"])
def test_importance_rules_bert_base(dev, rule):
    _full_check(wl.bert_base_bf16(), dev, 0.2, seed=0, importance=rule)


@pytest.mark.parametrize("rule", ["mean", "median"])
def test_importance_rules_single_token_row_and_eq6(dev, rule):
    # a row of one valid token (H len = H values), fp32, and the Eq. 6 probability
    L = wl.make_layer(3, 24, 64, 4, "f32", data_seed=9, lens=np.array([24, 1, 13]), q_scale=2.0,
                      token_scale_sigma=0.5)
    _full_check(L, dev, 0.1, seed=2, importance=rule)
    _full_check(L, dev, 0.1, seed=2, importance=rule, sampling="weight")


def _median_of(vals):
    """Median of float32 values as the median rule defines it: the middle value, or for an
    even count the mean of the two middle values taken in float64 and rounded once."""
    v = np.sort(vals.astype(np.float32))
    N = v.size
    lo, hi = v[(N - 1) // 2], v[N // 2]
    return np.float32(0.5 * (np.float64(lo) + np.float64(hi)))


@pytest.mark.parametrize("case", ["bert_base", "uniform", "small", "long"])
def test_median_selection_exact(dev, case):
    # the per-key median must be exactly the median of the probabilities the score pass
    # wrote (read back from the workspace), whichever selection path the column takes:
    # register select with compaction (BERT-base), without it (uniform attention: every
    # probability equal), eight registers (H len <= 512) and the LDS radix select
    # (H len > 2048)
    import torch

    import paper_2201_12854_amd as mca

    if case == "bert_base":
        L = wl.bert_base_bf16().subset([0, 1, 2])
    elif case == "uniform":
        L = wl.make_layer(2, 128, 96, 12, "bf16", data_seed=13, lens=np.array([128, 77]))
        L.Q[...] = 0.0
    elif case == "small":
        L = wl.make_layer(3, 40, 64, 4, "f32", data_seed=14, lens=np.array([40, 23, 1]), q_scale=2.0)
    else:
        L = wl.make_layer(2, 600, 128, 4, "bf16", data_seed=10, lens=np.array([600, 413]), q_scale=2.0)
    print(f"[case] median selection {case}: B={L.batch} n={L.seq} H={L.heads}", flush=True)
    t = to_device(L, dev)
    prep = mca.prepare_weights(t["Wv"])
    B, n, H = L.batch, L.seq, L.heads
    desc = mca.make_desc(B, n, H, L.d_in, 1 if L.dtype == "bf16" else 0, 0.4, 0,
                         importance=2)
    ws_bytes = mca.workspace_size(desc)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=dev)
    out = mca.attention_forward(t["Q"], t["K"], t["X"], t["Wv"], prep, 0.4, 0, heads=H, seq_lens=t["lens"],
                                export=True, workspace=ws, importance="median")
    torch.cuda.synchronize()
    acol_bytes = (4 * B * n * H * n + 255) // 256 * 256  # the last workspace segment
    acol = ws[ws_bytes - acol_bytes:ws_bytes - acol_bytes + 4 * B * n * H * n].view(torch.float32)
    acol = acol.reshape(B, n, H, n).cpu().numpy()
    m = out.colmax.cpu().numpy()
    for b in range(B):
        ln = int(L.lens[b])
        want = np.array([_median_of(acol[b, j, :, :ln].ravel()) for j in range(ln)])
        got = m[b, :ln]
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), \
            (b, np.flatnonzero(got != want)[:5])


# ------------------------------------------------------------------ exact encoding from a count
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("exact_from", [1, 20, 64])
def test_exact_from_small_ragged(dev, dtype, exact_from):
    # tokens with r >= exact_from take the exact MFMA path (in the gather for bf16, d_in
    # <= 768; in its own kernel for float32), the rest are sampled
    L = wl.make_layer(2, 40, 96, 4, dtype, data_seed=5, lens=np.array([40, 23]), q_scale=3.0,
                      token_scale_sigma=0.5)
    _full_check(L, dev, 0.4, seed=11, exact_from=exact_from)


def test_exact_from_bert_base_and_large(dev):
    _full_check(wl.bert_base_bf16(), dev, 0.4, seed=0, exact_from=128)
    _full_check(wl.make_layer(2, 300, 1024, 4, "bf16", data_seed=12, lens=np.array([300, 140]),
                              token_scale_sigma=0.5), dev, 0.2, seed=4, exact_from=96)


def test_forward_replays_from_a_captured_graph(dev):
    # the forward pass launches only kernels (no memset, no allocation), so a stream capture
    # replays it: three replays with eager work between them give the eager results bitwise
    import torch

    import paper_2201_12854_amd as mca

    L = wl.make_layer(4, 96, 256, 4, "bf16", data_seed=21, lens=np.array([96, 50, 1, 77]), q_scale=2.0,
                      token_scale_sigma=0.5)
    t = to_device(L, dev)
    prep = mca.prepare_weights(t["Wv"])
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        plan = mca.ForwardPlan(t["Q"], t["K"], t["X"], t["Wv"], prep, 0.4, 3, heads=L.heads, seq_lens=t["lens"])
        plan.run()
    torch.cuda.synchronize()
    Y0, r0 = plan.Y.clone(), plan.r.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        plan.run()
    for k in range(3):
        plan.Y.fill_(float("nan"))
        plan.r.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(plan.r, r0) and torch.equal(plan.Y, Y0), k
        with torch.cuda.stream(s):  # eager work between the replays
            plan.run()
        torch.cuda.synchronize()
        assert torch.equal(plan.Y, Y0)
