// Host-side launch interface of the MCA kernels (internal to libmca).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mca {

// Everything one forward pass needs, with the workspace already carved up.
struct FwdParams {
  int B, n, H, d_in, d_out;
  int bf16;  // 0: float32 inputs, 1: bfloat16 inputs
  double alpha;
  uint32_t seed_lo, seed_hi;
  const int32_t* seq_lens;  // [B] or null
  const int32_t* r_in;      // [B*n] or null
  const void* Q;
  const void* K;
  const void* X;
  const void* W;
  const float* rownorm;
  float* Y;
  int32_t* r;
  // workspace
  uint32_t* colmax_bits;  // [B*n]  float bits of m_j (non-negative, so uint order = float order)
  float* row_max;         // [B*H*n]
  float* row_inv_sum;     // [B*H*n]
  void* Henc;             // [B*n*d_out] H~ in bf16 (bf16 mode) or float32
  int32_t* sat_list;      // [B*n] tokens with r_j = d_in
  int32_t* counters;      // [4]; [0] = number of saturated tokens
  // optional outputs
  float* colmax_out;
  int32_t* idx_out;
  float* coef_out;
  float* enc_out;
};

hipError_t launch_clear(const FwdParams& p, hipStream_t s);
hipError_t launch_scores_colmax(const FwdParams& p, hipStream_t s);
hipError_t launch_encode(const FwdParams& p, hipStream_t s);
hipError_t launch_dense_encode(const FwdParams& p, hipStream_t s);
hipError_t launch_attn_out(const FwdParams& p, hipStream_t s);
hipError_t launch_rownorm(const void* W, int bf16, int d_in, int d_out, float* rownorm,
                          hipStream_t s);

// Dynamic LDS bytes of the encode kernel for (d_in, d_out).
size_t encode_lds_bytes(int d_in, int d_out);

}  // namespace mca
