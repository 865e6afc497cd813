// Exact encoding of saturated tokens (r_j = d_in): H~[j] = x_j W_v on MFMA.
//
// The count rule of Eq. 9 can ask for more samples than W_v has rows; such a token is
// encoded exactly, which costs what d_in samples would and has no error, so the error
// bounds of Lemma 1 / Theorem 1 still hold. The sampling kernel appends these tokens to
// a list; this kernel runs a [#saturated x d_in] x [d_in x d_out] GEMM over the list,
// 64 tokens x 64 columns per block (4 waves x 16 tokens). The grid covers the worst case
// (every token saturated) and blocks past the device-side count exit at once.
//   bf16: v_mfma_f32_16x16x32_bf16; the W_v tile is staged transposed in LDS so that each
//         lane's B operand (8 consecutive k of one column) is a single 16-byte read.
//   fp32: v_mfma_f32_16x16x4f32 with operands read straight from memory.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

constexpr int kThreads = 256;
constexpr int kTok = 64;
constexpr int kCols = 64;
constexpr int kKb = 32;               // k per staged bf16 W tile
constexpr int kWtStride = kKb + 8;    // LDS row stride (elements) of the transposed tile

template <int BF>
__device__ __forceinline__ void store_out(const FwdParams& p, int64_t off, float v) {
  if constexpr (BF) static_cast<uint16_t*>(p.Henc)[off] = (uint16_t)f32_to_bf16_bits(v);
  else static_cast<float*>(p.Henc)[off] = v;
  if (p.enc_out) p.enc_out[off] = v;
}

__global__ __launch_bounds__(kThreads) void k_dense_encode_bf16(FwdParams p) {
  __shared__ __align__(16) uint16_t Wt[kCols * kWtStride];  // [column][k]
  const int nsat = p.counters[0];
  const int t0 = blockIdx.x * kTok;
  if (t0 >= nsat) return;
  const int c0 = blockIdx.y * kCols;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in, d_out = p.d_out;
  const uint16_t* X = static_cast<const uint16_t*>(p.X);
  const uint16_t* W = static_cast<const uint16_t*>(p.W);

  const int slot = t0 + wave * 16 + r16;
  const int64_t tok = slot < nsat ? p.sat_list[slot] : -1;
  const uint16_t* xrow = X + (tok < 0 ? 0 : tok) * d_in;
  const bool xvec = (d_in & 7) == 0;

  f32x4_t acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < d_in; k0 += kKb) {
    __syncthreads();
    {  // W_v rows k0..k0+31, columns c0..c0+63 -> Wt[column][k]
      const int kr = tid >> 3, ch = tid & 7;
      uint4 u = make_uint4(0, 0, 0, 0);
      if (k0 + kr < d_in) u = *reinterpret_cast<const uint4*>(W + (int64_t)(k0 + kr) * d_out + c0 + 8 * ch);
      const uint32_t v[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Wt[(8 * ch + 2 * e) * kWtStride + kr] = (uint16_t)(v[e] & 0xffffu);
        Wt[(8 * ch + 2 * e + 1) * kWtStride + kr] = (uint16_t)(v[e] >> 16);
      }
    }
    __syncthreads();
    uint4 xa = make_uint4(0, 0, 0, 0);
    const int kx = k0 + 8 * g;
    if (tok >= 0) {
      if (xvec && kx + 8 <= d_in) {
        xa = *reinterpret_cast<const uint4*>(xrow + kx);
      } else {
        uint32_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) h[e] = (kx + e < d_in) ? xrow[kx + e] : 0u;
        xa = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
      }
    }
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, xa);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bf16x8_t bw = *reinterpret_cast<const bf16x8_t*>(Wt + (16 * c + r16) * kWtStride + 8 * g);
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bw, acc[c], 0, 0, 0);
    }
  }
  // acc[c][i] = H~[token slot 4 g + i of the wave][column c0 + 16 c + l % 16]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int sl = t0 + wave * 16 + 4 * g + i;
    if (sl < nsat) {
      const int64_t base = (int64_t)p.sat_list[sl] * d_out + c0 + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) store_out<1>(p, base + 16 * c, acc[c][i]);
    }
  }
}

__global__ __launch_bounds__(kThreads) void k_dense_encode_f32(FwdParams p) {
  const int nsat = p.counters[0];
  const int t0 = blockIdx.x * kTok;
  if (t0 >= nsat) return;
  const int c0 = blockIdx.y * kCols;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in, d_out = p.d_out;
  const float* X = static_cast<const float*>(p.X);
  const float* W = static_cast<const float*>(p.W);

  const int slot = t0 + wave * 16 + r16;
  const int64_t tok = slot < nsat ? p.sat_list[slot] : -1;
  const float* xrow = X + (tok < 0 ? 0 : tok) * d_in;
  const bool xvec = (d_in & 3) == 0;

  f32x4_t acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < d_in; k0 += 16) {
    // lane group g covers k = k0 + 4 g + t, t = 0..3 (the same k for both operands)
    const int kx = k0 + 4 * g;
    float xa[4];
    if (tok >= 0 && xvec && kx + 4 <= d_in) {
      const float4 v = *reinterpret_cast<const float4*>(xrow + kx);
      xa[0] = v.x; xa[1] = v.y; xa[2] = v.z; xa[3] = v.w;
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) xa[t] = (tok >= 0 && kx + t < d_in) ? xrow[kx + t] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const bool kval = kx + t < d_in;
      const float* wrow = W + (int64_t)(kval ? kx + t : 0) * d_out + c0 + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float bw = kval ? wrow[16 * c] : 0.f;
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[t], bw, acc[c], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int sl = t0 + wave * 16 + 4 * g + i;
    if (sl < nsat) {
      const int64_t base = (int64_t)p.sat_list[sl] * d_out + c0 + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) store_out<0>(p, base + 16 * c, acc[c][i]);
    }
  }
}

}  // namespace

hipError_t launch_dense_encode(const FwdParams& p, hipStream_t s) {
  const int64_t tokens = (int64_t)p.B * p.n;
  const dim3 grid((unsigned)((tokens + kTok - 1) / kTok), p.d_out / kCols);
  if (p.bf16) hipLaunchKernelGGL(k_dense_encode_bf16, grid, dim3(kThreads), 0, s, p);
  else hipLaunchKernelGGL(k_dense_encode_f32, grid, dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace mca
