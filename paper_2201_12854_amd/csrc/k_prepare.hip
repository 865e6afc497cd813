// One-time weight preparation (Sec. "Formulation of Sampling Probability": the per-row
// statistic of W is computed once per weight matrix and cached, not per forward pass):
//   rho_i = ||W_v[i, :]||, the row norms that scale the sampling weights of Eq. 4;
//   W_v^T in MFMA fragment order, the B operand of the MFMA products that encode saturated
//   tokens exactly (one coalesced 1 KB load per 16x16 tile and k step);
//   the sampling table of the paper's input-independent probability (Eq. 6), which
//   depends on W only: fixed-point weights of rho_i^2 and their prefix sums.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

// rho_i = float32(sqrt(sum_c W[i, c]^2)), float64 running sum in column order. A block of
// four waves per 64 rows: the waves load 64 x 64 tiles together (coalesced, the next tile
// in registers while the current one is summed) and wave 0 runs the 64 row sums, one row
// per lane, in column order.
template <int BF>
__global__ __launch_bounds__(256) void k_rownorm(const void* Wp, int d_in, int d_out, float* rownorm) {
  using T = typename Elem<BF>::T;
  __shared__ double tile[64][65];
  const T* W = static_cast<const T*>(Wp);
  const int r0 = blockIdx.x * 64, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  double nxt[16];
  auto load = [&](int c0) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int row = r0 + 16 * wave + j, c = c0 + lane;
      nxt[j] = (row < d_in && c < d_out) ? (double)load_f32(W, (int64_t)row * d_out + c) : 0.0;
    }
  };
  double s = 0.0;
  load(0);
  for (int c0 = 0; c0 < d_out; c0 += 64) {
#pragma unroll
    for (int j = 0; j < 16; ++j) tile[16 * wave + j][lane] = nxt[j];
    __syncthreads();
    if (c0 + 64 < d_out) load(c0 + 64);  // in flight during the sums
    if (wave == 0) {
      const int cend = min(64, d_out - c0);
      for (int cc = 0; cc < cend; ++cc) {
        const double v = tile[lane][cc];
        s = __dadd_rn(s, __dmul_rn(v, v));  // v*v is exact in float64
      }
    }
    __syncthreads();
  }
  if (wave == 0 && r0 + lane < d_in) rownorm[r0 + lane] = (float)sqrt(s);
}

// W_v^T in MFMA fragment order (layout in mca_kernels.h): one thread per 16-byte chunk;
// elements past d_in or d_out are zero. One-time preparation, so the strided reads of W
// are not tuned.
template <int BF>
__global__ __launch_bounds__(256) void k_fragment_wt(const void* Wp, int d_in, int d_out, int nks, int64_t nchunks,
                                                     void* Wtp) {
  using T = typename Elem<BF>::T;
  constexpr int E = BF ? 8 : 4, KS = 4 * E;
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= nchunks) return;
  const int l = (int)(q % 64);
  const int64_t tk = q / 64;  // t * nks + ks
  const int ks = (int)(tk % nks), t = (int)(tk / nks);
  const int c = 16 * t + (l % 16), k0 = ks * KS + (l / 16) * E;
  const T* W = static_cast<const T*>(Wp);
  T* dst = static_cast<T*>(Wtp) + q * E;
#pragma unroll
  for (int e = 0; e < E; ++e) dst[e] = (c < d_out && k0 + e < d_in) ? W[(int64_t)(k0 + e) * d_out + c] : T(0);
}

// Sampling table of the paper's input-independent probability (Eq. 6): v_i = fp32(rho_i^2),
// 32-bit fixed point aligned to the largest v_i, inclusive prefix sums. One block; each
// thread owns rows 2t and 2t + 1 (d_in <= 2048). All zero when every v_i is 0 or some v_i
// is not finite (no distribution: such tokens are encoded as 0).
__global__ __launch_bounds__(1024) void k_weight_table(const float* rownorm, int d_in, uint64_t* C) {
  __shared__ float smax[16];
  __shared__ uint64_t ssum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = 2 * tid;
  float v0 = 0.f, v1 = 0.f;
  if (i0 < d_in) v0 = __fmul_rn(rownorm[i0], rownorm[i0]);
  if (i0 + 1 < d_in) v1 = __fmul_rn(rownorm[i0 + 1], rownorm[i0 + 1]);
  // max with NaN ignored by fmaxf, so test finiteness on the values themselves
  const float lm = (v0 <= 3.40282347e38f && v1 <= 3.40282347e38f) ? fmaxf(v0, v1) : __int_as_float(0x7f800000);
  const float m = wave_max(lm);
  if (lane == 0) smax[wave] = m;
  __syncthreads();
  float vmax = smax[0];
#pragma unroll
  for (int w = 1; w < 16; ++w) vmax = fmaxf(vmax, smax[w]);
  if (!(vmax > 0.f) || !(vmax <= 3.40282347e38f)) {
    if (i0 < d_in) C[i0] = 0;
    if (i0 + 1 < d_in) C[i0 + 1] = 0;
    return;
  }
  int e;
  (void)frexpf(vmax, &e);  // vmax = f 2^e, f in [0.5, 1)
  const uint32_t w0 = i0 < d_in ? (uint32_t)ldexpf(v0, 32 - e) : 0u;
  const uint32_t w1 = i0 + 1 < d_in ? (uint32_t)ldexpf(v1, 32 - e) : 0u;
  const uint64_t s = (uint64_t)w0 + w1;
  uint64_t incl = s;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint64_t y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) ssum[wave] = incl;
  __syncthreads();
  uint64_t base = 0;
  for (int w = 0; w < wave; ++w) base += ssum[w];
  const uint64_t run = base + incl - s;
  if (i0 < d_in) C[i0] = run + w0;
  if (i0 + 1 < d_in) C[i0 + 1] = run + w0 + w1;
}

}  // namespace

hipError_t launch_prepare(const void* W, int bf16, int d_in, int d_out, void* prepared, hipStream_t s) {
  float* rownorm = static_cast<float*>(prepared);
  void* Wt = static_cast<char*>(prepared) + prepared_wt_offset(d_in);
  uint64_t* table = reinterpret_cast<uint64_t*>(static_cast<char*>(prepared) + prepared_table_offset(bf16, d_in, d_out));
  const int nks = (int)(prepared_din_pad(d_in) / (bf16 ? 32 : 16));
  const int64_t nchunks = prepared_dout_pad(d_out) / 16 * nks * 64;
  const dim3 g1((d_in + 63) / 64);
  const dim3 g2((unsigned)((nchunks + 255) / 256));
  if (bf16) {
    hipLaunchKernelGGL(k_rownorm<1>, g1, dim3(256), 0, s, W, d_in, d_out, rownorm);
    hipLaunchKernelGGL(k_fragment_wt<1>, g2, dim3(256), 0, s, W, d_in, d_out, nks, nchunks, Wt);
  } else {
    hipLaunchKernelGGL(k_rownorm<0>, g1, dim3(256), 0, s, W, d_in, d_out, rownorm);
    hipLaunchKernelGGL(k_fragment_wt<0>, g2, dim3(256), 0, s, W, d_in, d_out, nks, nchunks, Wt);
  }
  if (d_in > 2048) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_weight_table, dim3(1), dim3(1024), 0, s, rownorm, d_in, table);
  return hipGetLastError();
}

}  // namespace mca
