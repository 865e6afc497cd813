/*
 * mca.h - Monte-Carlo Attention (MCA) forward pass for AMD Instinct MI355X (gfx950).
 *
 * Kim & Ko, "Fast Monte-Carlo Approximation of the Attention Mechanism" (AAAI-22).
 * One attention layer Y = A (X W_v) (Eq. 1, Sec. "Self-Attention Mechanisms") in which
 * the encoding X W_v is replaced by the randomised estimator of Eq. 5: every token j
 * gets its own sample count r_j from the attention it receives (Eq. 9,
 * Sec. "Determining Sample Size from Attention") and is encoded with r_j importance
 * sampled rows of W_v (Eq. 2 with the optimal probability of Eq. 4).
 *
 * Plain C ABI: pointers, sizes and a stream handle; no C++ or framework types.
 *
 * Conventions shared by every entry point
 *  - "device" pointers point to memory of the current HIP device; "host" pointers to
 *    host memory. The caller owns every buffer; the library allocates no device memory
 *    and keeps no state between calls apart from optional profiler objects.
 *  - `stream` is a hipStream_t (NULL = the null stream). All device work is enqueued on
 *    it; nothing synchronises the host. Outputs are valid once the caller has
 *    synchronised the stream.
 *  - Arguments are checked on the host before anything is enqueued; a failed check
 *    returns a non-zero mca_status and enqueues nothing. mca_last_error() then gives a
 *    readable reason (thread-local). Nothing throws across this ABI and nothing aborts.
 *  - Layouts are row-major with the last index contiguous. Device pointers must be
 *    16-byte aligned.
 *  - Determinism: identical inputs, alpha and seed give bitwise-identical r, sample
 *    indices and Y.
 *  - Concurrent calls are safe when they use distinct workspaces and outputs.
 */
#ifndef MCA_H_
#define MCA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum mca_status {
  MCA_OK = 0,
  MCA_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad size, bad alpha, misalignment */
  MCA_ERR_UNSUPPORTED = 2,        /* valid, but outside what the kernels implement */
  MCA_ERR_WORKSPACE_TOO_SMALL = 3,
  MCA_ERR_HIP = 4                 /* a HIP runtime call or kernel launch failed */
} mca_status;

typedef enum mca_dtype {
  MCA_F32 = 0,   /* float32 inputs; fp32 MFMA and fp32 accumulation */
  MCA_BF16 = 1   /* bfloat16 inputs; bf16 MFMA with fp32 accumulation */
} mca_dtype;

/* Sampling probability of the encoding (Sec. "Formulation of Sampling Probability"). */
typedef enum mca_sampling {
  MCA_SAMPLING_TOKEN = 0,   /* Eq. 4 per token: p_ji proportional to |x_ji| * ||W_v[i, :]|| */
  MCA_SAMPLING_WEIGHT = 1   /* Eq. 6, input independent: p_i proportional to ||W_v[i, :]||^2
                               (the paper's own MCA); one distribution for every token */
} mca_sampling;

/* Stages of the forward pass, in launch order (profiler slots). */
typedef enum mca_importance {
  MCA_IMPORTANCE_MAX = 0,     /* m_j = max over valid queries and heads of A[:, j] (Eq. 8-9) */
  MCA_IMPORTANCE_MEAN = 1,    /* their mean */
  MCA_IMPORTANCE_MEDIAN = 2   /* their median (the mean of the two middle values for an even
                                 count); needs 4 B n H n bytes more workspace */
} mca_importance;

typedef enum mca_stage {
  MCA_STAGE_SCORES_COLMAX = 0,  /* softmax(Q K^T / 8) row statistics and column-max partials */
  MCA_STAGE_SAMPLE = 1,         /* count rule (Eq. 9), sampling weights (Eq. 4), draws, merge */
  MCA_STAGE_GATHER = 2,         /* H~: sampled rows gather-accumulate (and, for d_in <= 768 in
                                   bfloat16, the saturated tokens on MFMA) */
  MCA_STAGE_ATTN_OUT = 3,       /* Y = A H~ (MFMA) */
  MCA_STAGE_SATURATED = 4,      /* H~ = x W_v of the saturated tokens on MFMA, as a kernel of its
                                   own (d_in > 768 or float32 inputs; runs before the gather) */
  MCA_NUM_STAGES = 5
} mca_stage;

/*
 * Description of one forward call.
 *
 * Shapes: B = batch, n = seq (padded length), H = heads, d_head = 64,
 * d_out = H * 64, d_in = width of X.
 *   Q, K : [B, n, d_out], head h in columns h*64 .. h*64+63
 *   X    : [B, n, d_in]
 *   W_v  : [d_in, d_out]; row i belongs to input feature i (the X W convention of
 *          Eq. 1). A framework Linear weight [d_out, d_in] must be transposed.
 *   Y    : [B, n, d_out] float32
 *   r    : [B, n] int32
 */
typedef struct mca_forward_desc {
  int64_t batch;     /* B >= 1 */
  int64_t seq;       /* n >= 1 */
  int64_t heads;     /* H >= 1; d_out = 64 H must be a multiple of 256 and <= 2048 */
  int64_t d_head;    /* must be 64 (MCA_ERR_UNSUPPORTED otherwise) */
  int64_t d_in;      /* 1 .. 2048 */
  int32_t dtype;     /* mca_dtype of Q, K, X and W_v */
  int32_t sampling;  /* mca_sampling */
  double alpha;      /* attention error coefficient of Eq. 9; finite and > 0 */
  uint64_t seed;     /* Philox4x32-10 key (low word, high word) */
  /* device [B] int32 valid lengths (right padding), clamped to 1..n; NULL = all n */
  const int32_t* seq_lens;
  /* device [B*n] int32 or NULL. When set, replaces the count rule: token j of row b
     uses r_in[b*n+j] clamped to 0..d_in (padded keys still get 0). */
  const int32_t* r_in;
  /* Optional device outputs (NULL = not written):
     colmax_out      [B*n]       float32 m_j = max over heads and valid queries of A[:, j]
                                 (local window: of |S_i| A[i, j])
     sample_idx_out  [B*n*d_in]  int32: index s_k of draw k of token (b, j) at
                                 (b*n+j)*d_in + k, for k < r_j and 0 < r_j < d_in
     sample_coef_out [B*n*d_in]  float32 x_{s_k} T / (r_j w_{s_k}), same layout
     encoded_out     [B*n*d_out] float32 H~ (the estimated X W_v rows) */
  float* colmax_out;
  int32_t* sample_idx_out;
  float* sample_coef_out;
  float* encoded_out;
  /* mca_profiler handle from mca_profiler_create, or NULL. When set, the call records
     a pair of HIP events around every stage launch. */
  void* profiler;
  /* Attention pattern. 0: full attention. w > 0 (even): local window of w keys with a
     global first token (Sec. "Longformer": window 256, global attention for CLS):
     query i attends key j < len when |i - j| <= w / 2, or i = 0, or j = 0. The count
     rule then uses each query's key count |S_i| in place of n:
     m_j = max over heads and valid queries i of |S_i| A[i, j], t = m_j / alpha. */
  int64_t window;
  /* mca_importance: the per-key statistic m_j of the count rule under full attention
     (window = 0). MCA_IMPORTANCE_MAX is Eq. 8-9; the mean and the median are the more
     aggressive schemes the paper names after Eq. 8 (no error bound is proved for them). */
  int32_t importance;
  /* 0: tokens are encoded exactly (x_j W_v on MFMA) only when saturated (r_j = d_in).
     k > 0: also every token with r_j >= k, as its exact value costs less on the matrix
     cores than a long sampled list on the vector units (r_j is still reported). */
  int32_t exact_from;
} mca_forward_desc;

/*
 * Prepared weights: the per-row statistic of the value projection, computed once per
 * weight matrix and kept (Sec. "Formulation of Sampling Probability": it depends on W_v
 * only, so it need not be recomputed per input), plus a copy of W_v laid out for the
 * exact MFMA path.
 * Layout of the `prepared` buffer (device, caller-owned):
 *   offset 0:                        rownorm float32 [d_in]
 *                                    rownorm[i] = float32(sqrt(sum_c W_v[i, c]^2)), squares
 *                                    summed in float64 in column order c = 0 .. d_out-1, one
 *                                    IEEE square root, one rounding to float32 (bitwise
 *                                    reproducible)
 *   offset round_up(4 d_in, 256):    W_v^T in `dtype`, in MFMA fragment order: for column
 *                                    tile t (16 columns) and k step s (32 bf16 / 16 float32
 *                                    values of k), 64 x 16 bytes; the 16 bytes at index
 *                                    16 g + r hold W_v[s*KS + g*E + e][16 t + r], e < E
 *                                    (E = 8 bf16 / 4 float32); k zero padded to a multiple
 *                                    of 128, columns to a multiple of 16
 *   offset round_up(end of W_v^T, 256): uint64 [d_in] inclusive prefix sums C of the
 *                                    input-independent weights of Eq. 6: v_i =
 *                                    float32(rownorm[i] * rownorm[i]), w_i =
 *                                    floor(v_i 2^(32-e)) with max_i v_i = f 2^e, f in
 *                                    [0.5, 1); all zero when every v_i is 0 or one is
 *                                    not finite (then every sampled token encodes as 0)
 * mca_prepared_size gives the buffer size (host only). mca_prepare_weights fills it from
 * W_v (device [d_in, d_out] of `dtype`).
 * Errors: MCA_ERR_INVALID_ARGUMENT for null pointers, sizes < 1, d_in > 2048,
 * d_out > 1 << 20, a bad dtype, misalignment or prepared_bytes smaller than
 * mca_prepared_size; MCA_ERR_HIP if a launch fails.
 */
mca_status mca_prepared_size(int32_t dtype, int64_t d_in, int64_t d_out, size_t* bytes);
mca_status mca_prepare_weights(const void* W_v, int32_t dtype, int64_t d_in, int64_t d_out,
                               void* prepared, size_t prepared_bytes, void* stream);

/*
 * Bytes of device workspace mca_attention_forward needs for `desc` (host only, no
 * device work). Errors: as the argument checks of mca_attention_forward.
 */
mca_status mca_workspace_size(const mca_forward_desc* desc, size_t* bytes);

/*
 * One MCA forward pass (Eq. 5, with counts from Eq. 9):
 *   A_h   = softmax(Q_h K_h^T / 8), keys >= seq_lens[b] masked (and, with a local
 *           window, the keys outside each query's window)
 *   m_j   = max over heads h and valid queries i of A_h[i, j] (window: of |S_i| A_h[i, j])
 *   r_j   = min(max(ceil(t*t), 1), d_in), t = (len_b * m_j) / alpha in float64
 *           (window: t = m_j / alpha); 0 for padded keys. r_j = d_in marks a saturated
 *           token.
 *   H~[j] = (1/r_j) sum_k x_{j,s_k} W_v[s_k] / p(s_k)   for 0 < r_j < d_in
 *           with p(i) = w_i / T the 32-bit fixed-point form of |x_ji| * rownorm[i]
 *           (Eq. 4 for the product x_j W_v; MCA_SAMPLING_TOKEN) or of rownorm[i]^2
 *           (Eq. 6; MCA_SAMPLING_WEIGHT, from the prepared table), s_k drawn i.i.d. with replacement
 *           (Eq. 2) by Philox4x32-10 with key `seed` and counter (k, j, b, 0) and
 *           an inverse-CDF search; H~[j] = x_j W_v exactly when r_j = d_in; H~[j] = 0
 *           when r_j = 0, when x_j = 0 under Eq. 4, and when no distribution can be
 *           formed (all weights 0 or one of them not finite).
 *   Y_h   = A_h H~_h (per head column slice)
 * Inputs Q, K, X, W_v (device, `desc->dtype`) and `prepared` (filled by
 * mca_prepare_weights from this W_v with the same dtype and sizes). Outputs Y (device [B, n, d_out] float32) and r (device [B, n]
 * int32). Rows of Y for padded queries are computed by the same formula.
 * Q and K are expected to be finite: with a non-finite score, Y and r are unspecified
 * (every count stays in [0, d_in] and every access within the buffers).
 * `workspace` must hold at least mca_workspace_size bytes; its contents on entry do not
 * matter and are overwritten.
 * Errors: MCA_ERR_INVALID_ARGUMENT (null required pointer, size < 1, non-finite or
 * non-positive alpha, unknown sampling mode, odd or negative window, unknown importance rule or
 * a mean/median rule with a window, negative exact_from, misaligned pointer), MCA_ERR_UNSUPPORTED (d_head
 * != 64, d_out not a multiple of 256 or > 2048, d_in > 2048), MCA_ERR_WORKSPACE_TOO_SMALL,
 * MCA_ERR_HIP.
 */
mca_status mca_attention_forward(const mca_forward_desc* desc, const void* Q, const void* K,
                                 const void* X, const void* W_v, const void* prepared,
                                 float* Y, int32_t* r, void* workspace, size_t workspace_bytes,
                                 void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): mca_attention_forward without a
 * workspace argument. The scratch memory (column-max partials, row normalisers, H~ and the
 * sample lists) is a device array of MCA_NOALLOC_SCRATCH_BYTES inside the library, one per
 * device, held from the first call on that device until the process ends; the call itself
 * allocates nothing. Inputs, outputs and results are those of mca_attention_forward with
 * the same desc (the same kernels run).
 * Every call on a device shares that device's array and leaves its contents behind (the
 * kernels need none of them on entry): calls that overlap in time on one device (other
 * streams, other threads) race on it and must be serialised by the caller.
 * Errors: as mca_attention_forward, plus MCA_ERR_WORKSPACE_TOO_SMALL when
 * mca_workspace_size(desc) exceeds MCA_NOALLOC_SCRATCH_BYTES (then nothing is enqueued),
 * MCA_ERR_INVALID_ARGUMENT when desc->profiler is set (the profiler creates HIP events), and
 * MCA_ERR_HIP when the array's device address cannot be obtained.
 */
#define MCA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
mca_status mca_attention_forward_noalloc(const mca_forward_desc* desc, const void* Q, const void* K,
                                         const void* X, const void* W_v, const void* prepared,
                                         float* Y, int32_t* r, void* stream);

/* Static description of a status code (an mca_status value; any other value gives
   "MCA_ERR_UNKNOWN"). */
const char* mca_status_string(int status);

/* Reason for the last non-OK status returned on this thread ("" if none). */
const char* mca_last_error(void);

/* Number of forward stages (MCA_NUM_STAGES) and their names. */
int mca_num_stages(void);
const char* mca_stage_name(int stage);

/*
 * Per-stage kernel timing with HIP events, for benchmarks.
 * mca_profiler_create: *handle receives a new profiler (host object plus HIP events,
 *   created on the current device). MCA_ERR_HIP if event creation fails.
 * mca_profiler_collect: waits for every recorded event, then writes the summed
 *   milliseconds and the number of timed launches of each stage into stage_ms[0..n)
 *   and launches[0..n) (host arrays, n <= MCA_NUM_STAGES) and clears the records.
 * mca_profiler_destroy: releases the handle (NULL is accepted).
 * A profiler records at most 65536 stage launches between collections; further
 * launches run untimed.
 */
mca_status mca_profiler_create(void** handle);
mca_status mca_profiler_collect(void* handle, double* stage_ms, int64_t* launches, int n);
mca_status mca_profiler_destroy(void* handle);

#ifdef __cplusplus
}
#endif

#endif /* MCA_H_ */
