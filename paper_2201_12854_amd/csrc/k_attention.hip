// Attention stages of the MCA forward pass on gfx950:
//   scores + row softmax statistics + column max   (softmax(a Q K^T), a = 1/8, and the
//                                                    per-block part of max A[:, j], Eq. 8/9)
//   Y = A H~                                        ("Y = AH", Sec. "Self-Attention
//                                                    Mechanisms"; Eq. 5 outer sum)
// Both kernels rebuild the score tiles from Q and K with one shared routine, so the
// attention probabilities that set the sample counts are bitwise the ones multiplied
// into H~. A is never written to memory.
//
// Tiling: one block = 4 waves = 64 queries of one (batch row, head); a wave owns 16
// queries. Keys are processed in tiles of 64 staged in LDS. Scores are computed
// transposed, S^T = K Q^T, with 16x16 MFMA tiles (bf16 16x16x32 or fp32 16x16x4), so
// after the score MFMA lane l holds the scores of query (l % 16) for keys
// 16 s + 4 (l / 16) + i (s, i = 0..3): exactly the A-operand layout of the P V MFMA,
// with no data movement between the two products.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;                // queries per block and keys per tile
constexpr int kStrideBf = kDHead + 8;    // LDS row stride of bf16 tiles (elements)
constexpr int kStrideF = kDHead + 4;     // LDS row stride of fp32 tiles (elements)

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

// ------------------------------------------------------------------ Q fragments
// The wave's 16 queries as the B operand of S^T = K Q^T.
template <int BF> struct QFrag;
template <> struct QFrag<1> { bf16x8_t v[2]; };   // d = 32 ks + 8 g + (0..7)
template <> struct QFrag<0> { float v[16]; };      // d = 16 g + t

__device__ __forceinline__ void load_qfrag(QFrag<1>& f, const uint16_t* qrow, bool valid, int g) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (valid) u = *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g);
    f.v[ks] = __builtin_bit_cast(bf16x8_t, u);
  }
}

__device__ __forceinline__ void load_qfrag(QFrag<0>& f, const float* qrow, bool valid, int g) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float4 u = make_float4(0.f, 0.f, 0.f, 0.f);
    if (valid) u = *reinterpret_cast<const float4*>(qrow + 16 * g + 4 * c);
    f.v[4 * c + 0] = u.x;
    f.v[4 * c + 1] = u.y;
    f.v[4 * c + 2] = u.z;
    f.v[4 * c + 3] = u.w;
  }
}

// ------------------------------------------------------------------ LDS staging
// Rows key0 .. key0+63 of a [*, d_out] matrix (head column slice at `base`), rows >= n
// zero-filled, into a row-major LDS tile.
__device__ __forceinline__ void stage_rows(uint16_t* lds, const uint16_t* base, int64_t ld,
                                           int key0, int n, int tid) {
#pragma unroll
  for (int v = tid; v < kTile * 8; v += kThreads) {
    const int key = v >> 3, ch = v & 7;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (key0 + key < n) u = *reinterpret_cast<const uint4*>(base + (int64_t)(key0 + key) * ld + 8 * ch);
    *reinterpret_cast<uint4*>(lds + key * kStrideBf + 8 * ch) = u;
  }
}

__device__ __forceinline__ void stage_rows(float* lds, const float* base, int64_t ld, int key0,
                                           int n, int tid) {
#pragma unroll
  for (int v = tid; v < kTile * 16; v += kThreads) {
    const int key = v >> 4, ch = v & 15;
    float4 u = make_float4(0.f, 0.f, 0.f, 0.f);
    if (key0 + key < n) u = *reinterpret_cast<const float4*>(base + (int64_t)(key0 + key) * ld + 4 * ch);
    *reinterpret_cast<float4*>(lds + key * kStrideF + 4 * ch) = u;
  }
}

// bf16 H~ tile stored transposed ([column][key]) so that the B operand of the P V MFMA
// (8 keys of one column per lane) is two 8-byte LDS reads.
__device__ __forceinline__ void stage_rows_transposed(uint16_t* lds, const uint16_t* base, int64_t ld,
                                                      int key0, int n, int tid) {
#pragma unroll
  for (int v = tid; v < kTile * 8; v += kThreads) {
    const int key = v >> 3, ch = v & 7;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (key0 + key < n) u = *reinterpret_cast<const uint4*>(base + (int64_t)(key0 + key) * ld + 8 * ch);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lds[(8 * ch + 2 * e) * kStrideBf + key] = (uint16_t)(w[e] & 0xffffu);
      lds[(8 * ch + 2 * e + 1) * kStrideBf + key] = (uint16_t)(w[e] >> 16);
    }
  }
}

// ------------------------------------------------------------------ score tile
// acc[s][i] = (K Q^T)[key 16 s + 4 g + i][query l % 16] for the 64 keys in LDS.
__device__ __forceinline__ void score_tile(f32x4_t acc[4], const uint16_t* Ks, const QFrag<1>& q,
                                           int r16, int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    acc[s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(Ks + (16 * s + r16) * kStrideBf + 32 * ks + 8 * g);
      acc[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, q.v[ks], acc[s], 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void score_tile(f32x4_t acc[4], const float* Ks, const QFrag<0>& q,
                                           int r16, int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    acc[s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const float* krow = Ks + (16 * s + r16) * kStrideF + 16 * g;
#pragma unroll
    for (int t = 0; t < 16; ++t)
      acc[s] = __builtin_amdgcn_mfma_f32_16x16x4f32(krow[t], q.v[t], acc[s], 0, 0, 0);
  }
}

// Scaled logit a * (q . k) with a = 1/sqrt(64) = 1/8 (exact), kept free of contraction.
__device__ __forceinline__ float logit(float dot) { return __fmul_rn(dot, 0.125f); }

// Attention probability from the logit and the row statistics (max, 1/sum).
__device__ __forceinline__ float prob(float lg, float row_max, float row_inv) {
  return __fmul_rn(expf(__fsub_rn(lg, row_max)), row_inv);
}

__device__ __forceinline__ int valid_len(const FwdParams& p, int b) {
  int len = p.seq_lens ? p.seq_lens[b] : p.n;
  return min(max(len, 1), p.n);
}

// ------------------------------------------------------------------ kernels
template <int BF>
__global__ __launch_bounds__(kThreads) void k_scores_colmax(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int kStride = BF ? kStrideBf : kStrideF;
  __shared__ __align__(16) T Ks[kTile * kStride];
  __shared__ float cm[4][kTile];

  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int n = p.n, d_out = p.d_out, len = valid_len(p, b);
  const int q = qt * kTile + wave * 16 + r16;
  const T* Qb = static_cast<const T*>(p.Q) + (int64_t)b * n * d_out + h * kDHead;
  const T* Kb = static_cast<const T*>(p.K) + (int64_t)b * n * d_out + h * kDHead;

  QFrag<BF> qf;
  load_qfrag(qf, Qb + (int64_t)q * d_out, q < n, g);
  const int ntiles = (len + kTile - 1) / kTile;  // tiles past the valid length are all masked

  // Sweep 1: online row max and row sum of exp over the valid keys.
  float M = -INFINITY, L = 0.f;
  for (int kt = 0; kt < ntiles; ++kt) {
    lds_barrier();
    stage_rows(Ks, Kb, d_out, kt * kTile, n, tid);
    lds_barrier();
    f32x4_t acc[4];
    score_tile(acc, Ks, qf, r16, g);
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kt * kTile + 16 * s + 4 * g + i;
        const float lg = key < len ? logit(acc[s][i]) : -INFINITY;
        acc[s][i] = lg;
        mx = fmaxf(mx, lg);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float Mn = fmaxf(M, mx);
    float sum = 0.f;
    if (Mn != -INFINITY) {
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) sum += expf(__fsub_rn(acc[s][i], Mn));
    }
    sum += __shfl_xor(sum, 16, kWave);
    sum += __shfl_xor(sum, 32, kWave);
    L = (M == -INFINITY ? 0.f : __fmul_rn(L, expf(__fsub_rn(M, Mn)))) + sum;
    M = Mn;
  }
  const float inv = 1.0f / L;
  if (g == 0 && q < n) {
    const int64_t o = ((int64_t)b * p.H + h) * n + q;
    p.row_max[o] = M;
    p.row_inv_sum[o] = inv;
  }

  // Sweep 2: probabilities of valid queries and their max over this block's queries per
  // key, stored in this block's slot of the token's column-max partials (every slot is
  // written, so nothing needs clearing and no atomics are involved).
  const bool qvalid = q < len;
  float* part = p.colmax_part + (int64_t)b * n * p.nparts + h * p.qtiles + qt;
  for (int kt = 0; kt < ntiles; ++kt) {
    lds_barrier();
    stage_rows(Ks, Kb, d_out, kt * kTile, n, tid);
    lds_barrier();
    f32x4_t acc[4];
    score_tile(acc, Ks, qf, r16, g);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kt * kTile + 16 * s + 4 * g + i;
        float a = (qvalid && key < len) ? prob(logit(acc[s][i]), M, inv) : 0.f;
        a = fmaxf(a, __shfl_xor(a, 1, kWave));
        a = fmaxf(a, __shfl_xor(a, 2, kWave));
        a = fmaxf(a, __shfl_xor(a, 4, kWave));
        a = fmaxf(a, __shfl_xor(a, 8, kWave));
        if (r16 == 0) cm[wave][16 * s + 4 * g + i] = a;
      }
    lds_barrier();
    if (tid < kTile) {
      const float v = fmaxf(fmaxf(cm[0][tid], cm[1][tid]), fmaxf(cm[2][tid], cm[3][tid]));
      const int key = kt * kTile + tid;
      if (key < n) part[(int64_t)key * p.nparts] = v;
    }
  }
}

template <int BF>
__global__ __launch_bounds__(kThreads) void k_attn_out(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int kStride = BF ? kStrideBf : kStrideF;
  __shared__ __align__(16) T Ks[kTile * kStride];
  __shared__ __align__(16) T Vs[kTile * kStride];  // bf16: [column][key]; fp32: [key][column]

  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int n = p.n, d_out = p.d_out, len = valid_len(p, b);
  const int q = qt * kTile + wave * 16 + r16;
  const T* Qb = static_cast<const T*>(p.Q) + (int64_t)b * n * d_out + h * kDHead;
  const T* Kb = static_cast<const T*>(p.K) + (int64_t)b * n * d_out + h * kDHead;
  const T* Vb = static_cast<const T*>(p.Henc) + (int64_t)b * n * d_out + h * kDHead;

  QFrag<BF> qf;
  load_qfrag(qf, Qb + (int64_t)q * d_out, q < n, g);
  float M = 0.f, inv = 0.f;
  if (q < n) {
    const int64_t o = ((int64_t)b * p.H + h) * n + q;
    M = p.row_max[o];
    inv = p.row_inv_sum[o];
  }
  const int ntiles = (len + kTile - 1) / kTile;

  f32x4_t y[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) y[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt < ntiles; ++kt) {
    lds_barrier();
    stage_rows(Ks, Kb, d_out, kt * kTile, n, tid);
    if constexpr (BF) stage_rows_transposed(Vs, Vb, d_out, kt * kTile, n, tid);
    else stage_rows(Vs, Vb, d_out, kt * kTile, n, tid);
    lds_barrier();
    f32x4_t acc[4];
    score_tile(acc, Ks, qf, r16, g);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kt * kTile + 16 * s + 4 * g + i;
        acc[s][i] = key < len ? prob(logit(acc[s][i]), M, inv) : 0.f;
      }
    if constexpr (BF) {
      // 32 keys per MFMA: k-slots 0..3 = keys 32 pp + 4 g + (0..3), 4..7 = keys 32 pp + 16 + 4 g + (0..3)
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) {
        const uint4 pa = make_uint4(pack_bf16x2(acc[2 * pp][0], acc[2 * pp][1]),
                                    pack_bf16x2(acc[2 * pp][2], acc[2 * pp][3]),
                                    pack_bf16x2(acc[2 * pp + 1][0], acc[2 * pp + 1][1]),
                                    pack_bf16x2(acc[2 * pp + 1][2], acc[2 * pp + 1][3]));
        const bf16x8_t a = __builtin_bit_cast(bf16x8_t, pa);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint16_t* vrow = Vs + (16 * c + r16) * kStrideBf + 32 * pp + 4 * g;
          const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
          const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
          const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
          y[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bv, y[c], 0, 0, 0);
        }
      }
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float* vrow = reinterpret_cast<const float*>(Vs) + (16 * s + 4 * g + i) * kStrideF + r16;
#pragma unroll
          for (int c = 0; c < 4; ++c)
            y[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[s][i], vrow[16 * c], y[c], 0, 0, 0);
        }
    }
  }
  // y[c][i] = Y[query 4 g + i of the wave][column 16 c + l % 16]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = qt * kTile + wave * 16 + 4 * g + i;
    if (row < n) {
      float* yrow = p.Y + ((int64_t)b * n + row) * d_out + h * kDHead + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) yrow[16 * c] = y[c][i];
    }
  }
}

}  // namespace

hipError_t launch_scores_colmax(const FwdParams& p, hipStream_t s) {
  const dim3 grid((p.n + kTile - 1) / kTile, p.H, p.B);
  if (p.bf16) hipLaunchKernelGGL(k_scores_colmax<1>, grid, dim3(kThreads), 0, s, p);
  else hipLaunchKernelGGL(k_scores_colmax<0>, grid, dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_attn_out(const FwdParams& p, hipStream_t s) {
  const dim3 grid((p.n + kTile - 1) / kTile, p.H, p.B);
  if (p.bf16) hipLaunchKernelGGL(k_attn_out<1>, grid, dim3(kThreads), 0, s, p);
  else hipLaunchKernelGGL(k_attn_out<0>, grid, dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace mca
