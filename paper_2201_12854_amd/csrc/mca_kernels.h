// Host-side launch interface of the MCA kernels (internal to libmca).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mca {

constexpr int kQueryTile = 64;  // queries per attention block (the streaming kernels: 128)

// Queries per column-max partial: the query tile of the score pass, 128 for rows longer
// than 8 key tiles (its streaming kernel), else 64.
__host__ __device__ inline int score_query_tile(int n) { return (n + 63) / 64 > 8 ? 128 : 64; }


// Prepared weights: rownorm float32 [d_in] at offset 0, then, at prepared_wt_offset(d_in),
// W_v^T in the input dtype in MFMA fragment order: for every 16-column tile t and k step
// ks (KS = 32 bf16 or 16 float32 values of k), 64 lanes x 16 bytes, lane l = 16 g + r
// holding W_v[ks KS + g E + e][16 t + r], e < E (E = 8 bf16 or 4 float32 per 16 bytes).
// One wave-wide 16-byte load then fetches the B operand of a 16x16 MFMA tile as one
// contiguous 1 KB block. k is zero padded to a multiple of 128 (whole rounds of 4 steps),
// columns to a multiple of 16.
inline int64_t prepared_din_pad(int64_t d_in) { return (d_in + 127) / 128 * 128; }
inline int64_t prepared_dout_pad(int64_t d_out) { return (d_out + 15) / 16 * 16; }
inline size_t prepared_wt_offset(int64_t d_in) { return (size_t)((4 * d_in + 255) / 256 * 256); }
// Then, at prepared_table_offset, the input-independent sampling table of Eq. 6: uint64
// [d_in] inclusive prefix sums of the fixed-point weights of rho_i^2 (all zero when no
// distribution can be formed).
inline size_t prepared_table_offset(int bf16, int64_t d_in, int64_t d_out) {
  const size_t end = prepared_wt_offset(d_in) + (size_t)prepared_dout_pad(d_out) * (size_t)prepared_din_pad(d_in) * (bf16 ? 2 : 4);
  return (end + 255) / 256 * 256;
}
inline size_t prepared_bytes(int bf16, int64_t d_in, int64_t d_out) {
  return prepared_table_offset(bf16, d_in, d_out) + 8 * (size_t)d_in;
}

// Everything one forward pass needs, with the workspace already carved up.
struct FwdParams {
  int B, n, H, d_in, d_out;
  int bf16;     // 0: float32 inputs, 1: bfloat16 inputs
  int weight_sampling;  // 0: Eq. 4, p_ji ~ |x_ji| rho_i; 1: Eq. 6, p_i ~ rho_i^2
  int band_half;        // local window: query q attends keys within band_half of q and the
                        // first token attends and is attended by all (0: full attention)
  int importance;       // per-key statistic of the count rule: 0 max, 1 mean, 2 median
  int exact_from;       // > 0: tokens with r >= exact_from are encoded exactly too
  int qtiles;   // query tiles per sequence = ceil(n / score_query_tile(n))
  int nparts;   // column-max partials per token = H * qtiles
  int din_pad;  // row length of W_v^T
  double alpha;
  uint32_t seed_lo, seed_hi;
  const int32_t* seq_lens;  // [B] or null
  const int32_t* r_in;      // [B*n] or null
  const void* Q;
  const void* K;
  const void* X;
  const void* W;         // [d_in, d_out]
  const float* rownorm;  // [d_in]
  const void* Wt;        // W_v^T in MFMA fragment order
  const uint64_t* wtable;  // [d_in] Eq. 6 prefix sums
  float* Y;
  int32_t* r;
  // workspace
  float* colmax_part;  // [B*n][nparts]: max of A over one (head, query tile) block, per key
  float* acol;         // median rule: [B*n][H][n] A[h][query][key] per key (else null)
  float* row_c;        // [B*H*n] softmax normaliser of a query row in base-2 units:
                       // M + log2(sum of exp2(logit - M)), M the largest logit
  void* Henc;          // [B*n*d_out] H~ in the input dtype
  uint2* list;         // [B*n][list_stride(d_in)] distinct sampled rows of a token:
                       // (row * gather_row_bytes(d_in), float32 bits of coef); the even
                       // rows first, then the odd rows, each part padded to an even
                       // length with a zero row of its parity (rows d_in, d_in + 1 of the
                       // gather's LDS slice are zero)
  int32_t* ucount;     // [B*n] list layout of a sampled token: (even part length << 16) |
                       // total length; 0 when the token has no list
  int wc;              // W_v columns per gather slice (32 or 16)
  int sat_separate;    // saturated tokens encoded by their own kernel (the gather skips them)
  int gather_bps;      // gather blocks per slice
  // optional outputs
  float* colmax_out;
  int32_t* idx_out;
  float* coef_out;
  float* enc_out;
  // profiling: when set, the stage's kernel is launched with these events, which the
  // dispatch stamps at the kernel's start and end (kernel execution time only); a stage of
  // two kernels gives the start event to the first and the stop event to the second
  hipEvent_t ev_start, ev_stop;
};

// Launches a stage kernel, with the profiling events that are set.
template <typename K>
inline hipError_t launch_stage_kernel(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, const FwdParams& p) {
  if (p.ev_start || p.ev_stop) hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, p.ev_start, p.ev_stop, 0u, p);
  else hipLaunchKernelGGL(kernel, grid, block, lds, s, p);
  return hipGetLastError();
}

// A token encoded exactly (x_j W_v on MFMA) rather than sampled: saturated (r = d_in), or
// r >= exact_from when that is set.
__host__ __device__ inline bool exact_token(int r, int d_in, int exact_from) {
  return r >= d_in || (exact_from > 0 && r >= exact_from);
}

hipError_t launch_scores_colmax(const FwdParams& p, hipStream_t s);
hipError_t launch_sample(const FwdParams& p, hipStream_t s);
hipError_t launch_gather(const FwdParams& p, hipStream_t s);
// The exact encoding of saturated tokens as its own MFMA kernel (when sat_separate).
hipError_t launch_saturated(const FwdParams& p, hipStream_t s);
// Columns per gather slice for d_in (the slice, float32, must fit the LDS).
__host__ __device__ inline int gather_slice_cols(int d_in) { return d_in <= 1024 ? 32 : 16; }
// Entries reserved per token in the sample list: at most d_in - 1 distinct rows plus one
// pad entry per parity part, rounded up to even so that every list starts 16-byte aligned
// and entries can be read in pairs.
__host__ __device__ inline int list_stride(int d_in) { return (d_in + 2) & ~1; }
// Entries of slack after the last token's list: the gather kernel reads a few rounds past
// the end of a list (those entries are masked), which for the last tokens runs past
// their slots.
__host__ __device__ inline int list_tail_pad(int d_in) { return 2 * list_stride(d_in) + 64; }
// The two zero rows of the gather's LDS slice: even and odd row index.
__host__ __device__ inline int zero_row_even(int d_in) { return d_in + (d_in & 1); }
__host__ __device__ inline int zero_row_odd(int d_in) { return d_in + 1 - (d_in & 1); }
// Bytes of one slice row in LDS (float32); list entries hold row * gather_row_bytes.
__host__ __device__ inline int gather_row_bytes(int d_in) { return 4 * gather_slice_cols(d_in); }
// Gather blocks per column slice: at most one block per CU over all slices (a block holds
// most of a CU's LDS, so a second round of blocks would double the time).
int gather_blocks_per_slice(int d_in, int d_out);
hipError_t launch_attn_out(const FwdParams& p, hipStream_t s);
hipError_t launch_prepare(const void* W, int bf16, int d_in, int d_out, void* prepared, hipStream_t s);

}  // namespace mca
