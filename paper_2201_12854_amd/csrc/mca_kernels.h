// Host-side launch interface of the MCA kernels (internal to libmca).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mca {

constexpr int kQueryTile = 64;  // queries per attention block

// Prepared weights: rownorm float32 [d_in] at offset 0, then W_v^T [d_out][d_in_pad] in the
// input dtype (zero padded), at offset prepared_wt_offset(d_in).
inline int64_t prepared_din_pad(int64_t d_in) { return (d_in + 31) / 32 * 32; }
inline size_t prepared_wt_offset(int64_t d_in) { return (size_t)((4 * d_in + 255) / 256 * 256); }
inline size_t prepared_bytes(int bf16, int64_t d_in, int64_t d_out) {
  return prepared_wt_offset(d_in) + (size_t)d_out * (size_t)prepared_din_pad(d_in) * (bf16 ? 2 : 4);
}

// Everything one forward pass needs, with the workspace already carved up.
struct FwdParams {
  int B, n, H, d_in, d_out;
  int bf16;     // 0: float32 inputs, 1: bfloat16 inputs
  int qtiles;   // query tiles per sequence = ceil(n / kQueryTile)
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
  const void* Wt;        // [d_out, din_pad]
  float* Y;
  int32_t* r;
  // workspace
  float* colmax_part;  // [B*n][nparts]: max of A over one (head, query tile) block, per key
  float* row_max;      // [B*H*n]
  float* row_inv_sum;  // [B*H*n]
  void* Henc;          // [B*n*d_out] H~ in the input dtype
  // optional outputs
  float* colmax_out;
  int32_t* idx_out;
  float* coef_out;
  float* enc_out;
};

hipError_t launch_scores_colmax(const FwdParams& p, hipStream_t s);
hipError_t launch_encode(const FwdParams& p, hipStream_t s);
hipError_t launch_dense_encode(const FwdParams& p, hipStream_t s);
hipError_t launch_attn_out(const FwdParams& p, hipStream_t s);
hipError_t launch_prepare(const void* W, int bf16, int d_in, int d_out, void* prepared, hipStream_t s);

}  // namespace mca
