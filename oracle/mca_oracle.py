"""Plain CPU oracle of the Monte-Carlo Attention (MCA) forward pass, in float64.

TEST INFRASTRUCTURE ONLY. Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module. The product path (the
HIP library and its Python binding) never calls it and shares no code with it.

It follows Kim & Ko, "Fast Monte-Carlo Approximation of the Attention
Mechanism" (AAAI-22), step by step, in the paper's notation:

  O1  rho_i = ||W[i]||_2, cached once per weight matrix      (Sec. "Formulation of
      Sampling Probability": the per-row statistic depends on W only, so it is
      computed once and stored with the model)
  O2  A_h = softmax(a Q_h K_h^T), a = 1/sqrt(d_head)          (Sec. "Self-Attention
      Mechanisms", the definition of A before Eq. 1)
  O3  m_j = max A[:, j]  (largest attention key j receives,   (Sec. "Determining Sample
      over valid queries and all heads)                         Size from Attention", Eq. 8)
  O4  sqrt(r_j) = n * m_j / alpha                              (Eq. 9); m_j may instead be
      the mean or the median of A[:, j] (the more aggressive rules
      named after Eq. 8; no bound is proved for them)
  O5  p_ji proportional to |x_ji| * ||W[i]||                   (Eq. 4, the DKM-optimal
                                                                 probability, per token)
      or, in the paper's own input-independent mode,
      p_i proportional to ||W[i]||^2                           (Eq. 6, one distribution
                                                                 per weight matrix)
  O6  i.i.d. draws with replacement, Pr[s_k = i] = p(i)        (Eq. 2 and the text after it)
  O7  H~[j] = (1/r_j) sum_k x_{j,s_k} W[s_k] / p(s_k)          (Eq. 2 applied to X[j] W,
                                                                 i.e. Eq. 5's inner sum)
  O8  saturated tokens (r_j capped at d_in) are encoded exactly
  O9  Y~ = A H~, per head                                      (Eq. 5 / "Y = AH" of Eq. 1)

Local-window attention (Sec. "Longformer" and the document-classification
experiments: a window of w = 256 keys around each token plus global attention
for the first, CLS, token). With window w > 0, query i attends key j < len
when |i - j| <= w / 2, or i = 0, or j = 0; every other score is masked before
the softmax. The count rule follows the argument that leads to Eq. 9: the
error of row i sums over the |S_i| keys it attends (Eq. 8), so the factor n
that cancels that sum becomes |S_i|, and
  sqrt(r_j) = max over heads and valid queries i of |S_i| A[i, j] / alpha,
which is Eq. 9 when every row attends all n keys.

Readings taken where the paper is silent or garbled (each is listed with its
reason in the design notes of the repository):

* Eq. 5 indexes X[i, s_j[k]] inside the sum over tokens j; token j is encoded
  with its own samples, so the factor is X[j, s_j[k]].
* The count rule uses the number of *valid* tokens of the sequence as n, takes
  the ceiling of (n m_j / alpha)^2 in float64 in the order
  t = (n * m_j) / alpha; r = ceil(t * t), clamps it to [1, d_in], and gives
  padded keys r = 0. r_j = d_in marks a saturated token, encoded exactly.
* One r_j and one sample set per token, shared by all heads; m_j is the max
  over heads too.
* Finite-precision sampling distribution: v_i = fp32(|x_ji| * rho_i) (one
  IEEE float32 multiply), then 32-bit fixed-point weights
  w_i = floor(v_i * 2^(32 - e)) with v_max = f * 2^e, f in [0.5, 1). The
  distribution actually sampled is p^_i = w_i / T, T = sum_i w_i, and the
  estimator divides by p^_i, so it is exactly unbiased for
  sum_{w_i > 0} x_ji W[i].
* Random stream: Philox4x32-10 (Salmon et al., SC'11) with key
  (seed_lo, seed_hi) and counter (k, j, b, 0) for draw k of token j of batch
  row b; u = o0 | o1 << 32; t = floor(u * T / 2^64); s_k = min{i : C_i > t}
  with C the inclusive prefix sums of w.
* A token whose weights are all zero (x_j = 0) is encoded as 0.
* Local-window mode: w / 2 keys on each side (w even), the first token global
  in both directions; m_j is the largest |S_i| A[i, j] (float64) and
  t = m_j / alpha, r = ceil(t * t) clamped as above. With w = 0 (full
  attention) the rule is the one printed, t = (n * m_j) / alpha.
* Eq. 6 mode: v_i = fp32(rho_i * rho_i) (one IEEE float32 multiply of the
  float32 row norm), then the same fixed-point weights, prefix sums, random
  stream and inverse CDF. The table depends on W only, so it is built once and
  every token draws from it; a token with x_j = 0 still draws, with
  coefficients 0, so its H~[j] is 0.
"""
from __future__ import annotations

import bisect
import math

import numpy as np

D_HEAD = 64
MASK32 = 0xFFFFFFFF

SAMPLING_TOKEN = "token"    # Eq. 4: p_ji proportional to |x_ji| ||W[i]||
SAMPLING_WEIGHT = "weight"  # Eq. 6: p_i proportional to ||W[i]||^2

# Philox4x32 constants as published by Salmon, Moraes, Dror and Shaw,
# "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11): two round multipliers
# and the two Weyl-sequence key increments (golden ratio, sqrt(3) - 1).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
PHILOX_ROUNDS = 10


# --------------------------------------------------------------------------- O6 RNG
def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds, vectorised over numpy arrays.

    ``ctr`` is four arrays (or ints) of 32-bit counter words, ``key`` two
    32-bit key words. Each round multiplies counter words 0 and 2 by the two
    round constants (64-bit products), and outputs
    (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));
    the key is advanced by the Weyl increments between rounds.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & np.uint64(MASK32) for c in ctr)
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for _ in range(PHILOX_ROUNDS):
        p0 = np.uint64(PHILOX_M0) * c0  # < 2^64: exact
        p1 = np.uint64(PHILOX_M1) * c2
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ np.uint64(k0),
                          p1 & np.uint64(MASK32),
                          (p0 >> np.uint64(32)) ^ c3 ^ np.uint64(k1),
                          p0 & np.uint64(MASK32))
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return c0, c1, c2, c3


def uniform_u64(seed: int, b: int, j: int, ks) -> list:
    """64-bit uniform words for draws ``ks`` of token j in batch row b."""
    ks = np.asarray(ks, dtype=np.uint64)
    zero = np.zeros_like(ks)
    o0, o1, _, _ = philox4x32_10((ks, zero + np.uint64(j), zero + np.uint64(b), zero),
                                 (seed & MASK32, (seed >> 32) & MASK32))
    return [int(a) | (int(c) << 32) for a, c in zip(o0.tolist(), o1.tolist())]


# --------------------------------------------------------------------------- O1
def row_norms(W: np.ndarray) -> np.ndarray:
    """rho_i = fp32(sqrt(sum_c W[i, c]^2)): float64 squares summed in column order
    c = 0, 1, ... (a sequential running sum), IEEE sqrt, then one rounding to
    float32. Row i of W is input feature i (the X W convention of Eq. 1)."""
    sq = np.asarray(W, dtype=np.float64) ** 2
    running = np.cumsum(sq, axis=1)  # sequential accumulation, left to right
    return np.sqrt(running[:, -1]).astype(np.float32)


# --------------------------------------------------------------------------- O2
def attended(q_pos, n_keys: int, valid: int, window: int = 0) -> np.ndarray:
    """Boolean [len(q_pos), n_keys]: query at position q attends key j. Keys at or
    past ``valid`` are padding. window = 0: every valid key (full attention);
    window w > 0: |q - j| <= w / 2, plus the global first token (query 0 attends
    every valid key and every query attends key 0)."""
    q = np.asarray(q_pos, dtype=np.int64)[:, None]
    j = np.arange(n_keys, dtype=np.int64)[None, :]
    ok = np.broadcast_to(j < valid, (q.shape[0], n_keys))
    if window > 0:
        ok = ok & ((np.abs(q - j) <= window // 2) | (q == 0) | (j == 0))
    return ok


def attention_probs(Qbh: np.ndarray, Kbh: np.ndarray, valid: int, window: int = 0, q0: int = 0) -> np.ndarray:
    """A = softmax(a Q K^T) with a = 1/sqrt(d_head), over the keys each query attends
    (``attended``; the rows of Qbh are the queries at positions q0, q0 + 1, ...);
    every other key gets probability 0. Rows of padded queries are computed the
    same way (they are not used for the counts)."""
    Q = np.asarray(Qbh, dtype=np.float64)
    K = np.asarray(Kbh, dtype=np.float64)
    S = (Q @ K.T) * (1.0 / math.sqrt(Q.shape[1]))
    S[~attended(np.arange(q0, q0 + Q.shape[0]), K.shape[0], valid, window)] = -np.inf
    S = S - S.max(axis=1, keepdims=True)
    E = np.exp(S)
    return E / E.sum(axis=1, keepdims=True)


def head_slice(h: int) -> slice:
    return slice(h * D_HEAD, (h + 1) * D_HEAD)


# --------------------------------------------------------------------------- O3
def keys_attended(valid: int, window: int = 0) -> np.ndarray:
    """|S_i| for the valid queries i < valid: how many keys each one attends."""
    return attended(np.arange(valid), valid, valid, window).sum(axis=1)


def column_max(Q, K, lens, heads, window: int = 0) -> np.ndarray:
    """m[b, j] = max over heads h and valid queries i of A_h[b, i, j] (window 0), or of
    |S_i| A_h[b, i, j] (window > 0, the count rule's per-row factor); 0 for padded keys."""
    B, n = Q.shape[0], Q.shape[1]
    m = np.zeros((B, n), dtype=np.float64)
    for b in range(B):
        L = int(lens[b])
        scale = keys_attended(L, window).astype(np.float64)[:, None] if window > 0 else 1.0
        for h in range(heads):
            A = attention_probs(Q[b, :, head_slice(h)], K[b, :, head_slice(h)], L, window)
            m[b] = np.maximum(m[b], (scale * A[:L]).max(axis=0))
        m[b, L:] = 0.0
    return m


IMPORTANCE_MAX = "max"        # Eq. 8-9: the largest attention a key receives
IMPORTANCE_MEAN = "mean"      # the mean over valid queries and heads (a more aggressive rule)
IMPORTANCE_MEDIAN = "median"  # the median over valid queries and heads


def column_importance(Q, K, lens, heads, rule: str = IMPORTANCE_MAX) -> np.ndarray:
    """The per-key statistic that sets the count under full attention: the max of
    A_h[b, i, j] over heads h and valid queries i (Eq. 8-9), or, as the more aggressive
    schemes the paper names after Eq. 8, their mean or median (over the H * len values;
    for an even count the median is the mean of the two middle values). 0 for padded
    keys."""
    if rule == IMPORTANCE_MAX:
        return column_max(Q, K, lens, heads)
    if rule not in (IMPORTANCE_MEAN, IMPORTANCE_MEDIAN):
        raise ValueError(f"unknown importance rule {rule!r}")
    B, n = Q.shape[0], Q.shape[1]
    m = np.zeros((B, n), dtype=np.float64)
    for b in range(B):
        L = int(lens[b])
        vals = np.stack([attention_probs(Q[b, :, head_slice(h)], K[b, :, head_slice(h)], L)[:L, :L]
                         for h in range(heads)])  # [H, queries, keys]
        per_key = vals.transpose(2, 0, 1).reshape(L, heads * L)
        m[b, :L] = per_key.mean(axis=1) if rule == IMPORTANCE_MEAN else np.median(per_key, axis=1)
    return m


# --------------------------------------------------------------------------- O4
def sample_counts(m: np.ndarray, lens, alpha: float, d_in: int, window: int = 0) -> np.ndarray:
    """Eq. 9: sqrt(r_j) = n * m_j / alpha with n the valid length of the sequence;
    r_j = min(max(ceil(t*t), 1), d_in) with t = (n*m_j)/alpha in float64;
    padded keys get 0. Window mode: m_j already carries the per-row factor
    |S_i|, so t = m_j / alpha."""
    B, n = m.shape
    r = np.zeros((B, n), dtype=np.int64)
    for b in range(B):
        L = int(lens[b])
        for j in range(L):
            t = (float(m[b, j]) if window > 0 else float(L) * float(m[b, j])) / float(alpha)
            tt = t * t
            r[b, j] = min(max(math.ceil(tt), 1), d_in) if math.isfinite(tt) else d_in
    return r


# --------------------------------------------------------------------------- O5
def quantise(v: np.ndarray):
    """32-bit fixed point of non-negative float32 values: e such that
    v_max = f * 2^e, f in [0.5, 1); w_i = floor(v_i * 2^(32-e)) (exact: a
    power-of-two scaling of a float32 value in float64). Returns (w as Python
    ints, inclusive prefix sums C, total T), or None when every v_i is 0 or some
    v_i is not finite (a float32 overflow of |x_i| rho_i or rho_i^2): such a
    token has no usable distribution and is encoded as 0."""
    vmax = float(v.max()) if v.size else 0.0
    if vmax == 0.0 or not math.isfinite(vmax):
        return None
    _, e = math.frexp(vmax)
    w = [int(math.floor(math.ldexp(float(vi), 32 - e))) for vi in v]
    C = []
    acc = 0
    for wi in w:
        acc += wi
        C.append(acc)
    return w, C, acc


def fixed_point_weights(x: np.ndarray, rho: np.ndarray):
    """Integer sampling weights of one token (Eq. 4 with B = W: p_i is proportional
    to |x_i| * ||W[i]||): v_i = fp32(|x_i| * rho_i), quantised."""
    v = np.abs(np.asarray(x, dtype=np.float32)) * np.asarray(rho, dtype=np.float32)
    return quantise(v.astype(np.float32))


def weight_fixed_point(rho: np.ndarray):
    """Integer sampling weights of the paper's input-independent distribution
    (Eq. 6: p_i = ||W[i]||^2 / ||W||_F^2): v_i = fp32(rho_i * rho_i), quantised.
    One table per weight matrix."""
    r32 = np.asarray(rho, dtype=np.float32)
    return quantise((r32 * r32).astype(np.float32))


def index_from_u(u: int, C, T: int) -> int:
    """Inverse CDF: t = floor(u T / 2^64) in [0, T); the index is the smallest i with C_i > t."""
    t = (u * T) >> 64
    return bisect.bisect_right(C, t)


def draw_indices(C, T: int, r: int, seed: int, b: int, j: int) -> list:
    """r i.i.d. indices with Pr[s = i] = w_i / T (Eq. 2: sampling with replacement)."""
    if r <= 0:
        return []
    return [index_from_u(u, C, T) for u in uniform_u64(seed, b, j, np.arange(r))]


# --------------------------------------------------------------------------- O7
def coefficients(x: np.ndarray, w, T: int, idx, r: int) -> np.ndarray:
    """Per-sample scale x_{s_k} / (r p^(s_k)) = x_{s_k} T / (r w_{s_k}) of Eq. 2."""
    return np.array([float(x[s]) * float(T) / (float(r) * float(w[s])) for s in idx],
                    dtype=np.float64)


def estimate_from_indices(x: np.ndarray, W: np.ndarray, w, T: int, idx, r: int) -> np.ndarray:
    """Eq. 2 for the product X[j] W: (1/r) sum_k x_{s_k} W[s_k] / p^(s_k)."""
    W64 = np.asarray(W, dtype=np.float64)
    out = np.zeros(W64.shape[1], dtype=np.float64)
    for c, s in zip(coefficients(x, w, T, idx, r), idx):
        out += c * W64[s]
    return out


def encode_token(x, W, rho, r: int, seed: int, b: int, j: int, *, sampling=SAMPLING_TOKEN, table=None,
                 exact_from: int = 0):
    """H~[j] for one token. Returns (H~[j], indices, coefficients). In Eq. 6 mode
    ``table`` is weight_fixed_point(rho) (computed here when not given). ``exact_from``
    > 0 encodes every token with r >= exact_from exactly as well (no draws)."""
    d_in = W.shape[0]
    if r <= 0:
        return np.zeros(W.shape[1]), [], np.zeros(0)
    if r >= d_in or (exact_from > 0 and r >= exact_from):  # O8: saturated, exact encoding
        return np.asarray(x, np.float64) @ np.asarray(W, np.float64), [], np.zeros(0)
    if sampling == SAMPLING_WEIGHT:
        fp = table if table is not None else weight_fixed_point(rho)
    else:
        fp = fixed_point_weights(x, rho)
    if fp is None:  # all-zero token (Eq. 4) or all-zero W (Eq. 6)
        return np.zeros(W.shape[1]), [], np.zeros(0)
    w, C, T = fp
    idx = draw_indices(C, T, r, seed, b, j)
    coef = coefficients(x, w, T, idx, r)
    W64 = np.asarray(W, dtype=np.float64)
    H = coef @ W64[idx] if idx else np.zeros(W.shape[1])
    return H, idx, coef


# --------------------------------------------------------------------------- forward
def mca_forward(Q, K, X, W, lens, heads: int, alpha: float, seed: int, *, r_override=None,
                rho=None, y_rows=None, want_samples=False, want_exact=False, sampling=SAMPLING_TOKEN,
                window: int = 0, importance: str = IMPORTANCE_MAX, exact_from: int = 0):
    """Full MCA forward (O1-O9) for right-padded sequences.

    Q, K: [B, n, heads*64]; X: [B, n, d_in]; W: [d_in, heads*64] (all float32
    holding the layer's values). ``r_override`` replaces the count rule (O4);
    padded keys still get 0. ``y_rows`` restricts the output to selected
    (b, i) query rows (the counts and encodings are always computed for all
    tokens, because every query row depends on all of them).
    Returns a dict with rho, m, r, Htilde, Y (or Y at y_rows), and optionally
    samples (per token: indices, coefficients) and the exact Y* of Eq. 1.
    ``sampling`` selects the probability: SAMPLING_TOKEN (Eq. 4, per token) or
    SAMPLING_WEIGHT (Eq. 6, one table per weight matrix). ``window`` > 0 selects
    local-window attention with a global first token (see ``attended``). ``importance``
    selects the per-key statistic of the count rule (``column_importance``; full
    attention only for the mean and median). ``exact_from`` > 0: tokens whose count
    reaches it are encoded exactly, like saturated ones (their counts are still reported;
    0 keeps exact encoding for r = d_in only, the paper's case).
    """
    if window < 0 or window % 2:
        raise ValueError("window must be 0 (full attention) or a positive even number of keys")
    if importance != IMPORTANCE_MAX and window:
        raise ValueError("the mean and median rules are defined for full attention")
    if exact_from < 0:
        raise ValueError("exact_from must be >= 0")
    B, n, d_in = X.shape
    d_out = W.shape[1]
    lens = np.asarray(lens)
    if rho is None:
        rho = row_norms(W)
    m = column_max(Q, K, lens, heads, window) if importance == IMPORTANCE_MAX else \
        column_importance(Q, K, lens, heads, importance)
    if r_override is None:
        r = sample_counts(m, lens, alpha, d_in, window)
    else:
        r = np.array(r_override, dtype=np.int64).reshape(B, n).copy()
        r = np.clip(r, 0, d_in)
        for b in range(B):
            r[b, int(lens[b]):] = 0
    if sampling not in (SAMPLING_TOKEN, SAMPLING_WEIGHT):
        raise ValueError(f"unknown sampling mode {sampling!r}")
    table = weight_fixed_point(rho) if sampling == SAMPLING_WEIGHT else None
    Ht = np.zeros((B, n, d_out), dtype=np.float64)
    samples = {}
    for b in range(B):
        for j in range(n):
            H, idx, coef = encode_token(X[b, j], W, rho, int(r[b, j]), seed, b, j, sampling=sampling, table=table,
                                        exact_from=exact_from)
            Ht[b, j] = H
            if want_samples:
                samples[(b, j)] = (idx, coef)
    out = {"rho": rho, "m": m, "r": r, "Htilde": Ht}
    Hx = None
    if want_exact:
        Hx = np.asarray(X, np.float64) @ np.asarray(W, np.float64)
    if y_rows is None:
        Y = np.zeros((B, n, d_out))
        Yx = np.zeros((B, n, d_out)) if want_exact else None
        for b in range(B):
            for h in range(heads):
                cs = head_slice(h)
                A = attention_probs(Q[b, :, cs], K[b, :, cs], int(lens[b]), window)
                Y[b, :, cs] = A @ Ht[b, :, cs]
                if want_exact:
                    Yx[b, :, cs] = A @ Hx[b, :, cs]
        out["Y"] = Y
        if want_exact:
            out["Yexact"] = Yx
    else:
        rows = [(int(b), int(i)) for b, i in y_rows]
        Y = np.zeros((len(rows), d_out))
        for t, (b, i) in enumerate(rows):
            for h in range(heads):
                cs = head_slice(h)
                A = attention_probs(Q[b, i:i + 1, cs], K[b, :, cs], int(lens[b]), window, q0=i)
                Y[t, cs] = A[0] @ Ht[b, :, cs]
        out["Y_rows"] = Y
    if want_samples:
        out["samples"] = samples
    return out


def exact_forward(Q, K, X, W, lens, heads: int, window: int = 0) -> np.ndarray:
    """Eq. 1: Y[i] = sum_j A[i, j] X[j] W, per head, in float64."""
    B, n, _ = X.shape
    H = np.asarray(X, np.float64) @ np.asarray(W, np.float64)
    Y = np.zeros((B, n, W.shape[1]))
    for b in range(B):
        for h in range(heads):
            cs = head_slice(h)
            A = attention_probs(Q[b, :, cs], K[b, :, cs], int(lens[b]), window)
            Y[b, :, cs] = A @ H[b, :, cs]
    return Y


# --------------------------------------------------------------------------- closed forms
def estimator_variance(x, W, w, T: int, r: int) -> float:
    """E||H~ - E H~||^2 for the quantised distribution p^_i = w_i / T:
    (1/r) (T sum_{w_i>0} x_i^2 ||W[i]||^2 / w_i - ||sum_{w_i>0} x_i W[i]||^2)."""
    W64 = np.asarray(W, np.float64)
    x64 = np.asarray(x, np.float64)
    keep = [i for i, wi in enumerate(w) if wi > 0]
    first = sum(x64[i] ** 2 * float(W64[i] @ W64[i]) * T / w[i] for i in keep)
    mean = sum((x64[i] * W64[i] for i in keep), np.zeros(W64.shape[1]))
    return (first - float(mean @ mean)) / r
