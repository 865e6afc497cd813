// Sampled value encoding of the MCA forward pass on gfx950.
//
// One block (4 waves) per token j of batch row b:
//   1. sample count r_j from the column max (Eq. 9, Sec. "Determining Sample Size
//      from Attention"), in float64: t = (len_b * m_j) / alpha, r_j = ceil(t * t)
//      clamped to [1, d_in]; padded keys get 0; r_j = d_in hands the token to the
//      exact MFMA path.
//   2. sampling weights of Eq. 4 for the product x_j W_v: v_i = |x_ji| * rho_i in one
//      float32 multiply, quantised to 32-bit fixed point aligned to the largest v_i,
//      w_i = floor(v_i 2^(32-e)); inclusive prefix sums C (uint64) in LDS.
//   3. r_j i.i.d. draws with replacement (Eq. 2): Philox4x32-10 with counter
//      (k, j, b, 0), u = o0 | o1 << 32, t = floor(u T / 2^64), s_k = min{i : C_i > t}
//      by binary search in LDS. Draws are counted per row with LDS integer atomics
//      (exact, order-free).
//   4. duplicates merged: coefficient of row i = count_i x_ji T / (r_j w_i) (float64,
//      rounded once), rows compacted in ascending order.
//   5. gather-scale-accumulate: each wave streams a quarter of the distinct rows of W_v
//      with coalesced vector loads and accumulates in float32; the four partial rows
//      are summed in a fixed order through LDS.
// Everything is deterministic: the same inputs and seed give bitwise-equal output.
//
// Also here: the one-time row-norm kernel (Sec. "Formulation of Sampling Probability":
// the per-row statistic of W is computed once and cached).
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

struct EncodeLds {
  int off_C, off_w, off_cnt, off_uidx, off_ucoef, off_misc, total;
};

__host__ __device__ inline int round_up(int v, int a) { return (v + a - 1) / a * a; }

__host__ __device__ inline EncodeLds encode_lds_layout(int d_in, int d_out) {
  EncodeLds l;
  l.off_C = 0;                       // uint64 [d_in]
  l.off_w = 8 * d_in;                // uint32 [d_in]
  l.off_cnt = 12 * d_in;             // uint32 [d_in]
  // the partial-row reduction buffer float [4][d_out] aliases C, w and cnt
  const int region0 = round_up(16 * (d_in > d_out ? d_in : d_out), 16);
  l.off_uidx = region0;              // int32 [d_in]
  l.off_ucoef = region0 + 4 * d_in;  // float [d_in]
  l.off_misc = round_up(region0 + 8 * d_in, 16);
  l.total = l.off_misc + 64;
  return l;
}

// Writes one H~ row (4 consecutive columns per call).
template <int BF> struct HStore;
template <> struct HStore<1> {
  static __device__ __forceinline__ void store(void* H, int64_t off, float4 v) {
    uint2 u = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(H) + off) = u;
  }
};
template <> struct HStore<0> {
  static __device__ __forceinline__ void store(void* H, int64_t off, float4 v) {
    *reinterpret_cast<float4*>(static_cast<float*>(H) + off) = v;
  }
};

template <int BF>
__device__ __forceinline__ void write_row(const FwdParams& p, int64_t tok, float4 v, int c) {
  const int64_t off = tok * p.d_out + c;
  HStore<BF>::store(p.Henc, off, v);
  if (p.enc_out) *reinterpret_cast<float4*>(p.enc_out + off) = v;
}

template <int BF>
__device__ void write_zero_row(const FwdParams& p, int64_t tok, int tid) {
  for (int c = 4 * tid; c < p.d_out; c += 4 * kThreads) write_row<BF>(p, tok, make_float4(0.f, 0.f, 0.f, 0.f), c);
}

// Exclusive prefix (over the block, thread order) of a per-thread value; also returns
// the block total. `scratch` holds kWaves values. Contains __syncthreads.
template <typename U>
__device__ __forceinline__ U block_exclusive_scan(U v, U* scratch, U* total, int lane, int wave) {
  U incl = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const U y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) scratch[wave] = incl;
  __syncthreads();
  U base = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) base += scratch[w];
    all += scratch[w];
  }
  *total = all;
  return base + incl - v;
}

template <int BF, int NV>
__global__ __launch_bounds__(kThreads) void k_encode(FwdParams p) {
  using T = typename Elem<BF>::T;
  extern __shared__ __align__(16) unsigned char smem[];
  const int d_in = p.d_in, d_out = p.d_out, n = p.n;
  const int64_t tok = blockIdx.x;
  const int b = (int)(tok / n), j = (int)(tok - (int64_t)b * n);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int len = p.seq_lens ? p.seq_lens[b] : n;
  len = min(max(len, 1), n);

  // ---- 1. sample count (Eq. 9)
  int r;
  if (j >= len) {
    r = 0;
  } else if (p.r_in) {
    r = min(max(p.r_in[tok], 0), d_in);
  } else {
    const float m = __uint_as_float(p.colmax_bits[tok]);
    const double t = ((double)len * (double)m) / p.alpha;
    const double tt = t * t;
    r = (tt >= (double)d_in) ? d_in : max((int)ceil(tt), 1);
  }
  if (tid == 0) {
    p.r[tok] = r;
    if (p.colmax_out) p.colmax_out[tok] = __uint_as_float(p.colmax_bits[tok]);
  }
  if (r == 0) {
    write_zero_row<BF>(p, tok, tid);
    return;
  }
  if (r >= d_in) {  // saturated: exact encoding by the MFMA path
    if (tid == 0) {
      const int pos = atomicAdd(p.counters, 1);
      p.sat_list[pos] = (int32_t)tok;
    }
    return;
  }

  const EncodeLds L = encode_lds_layout(d_in, d_out);
  uint64_t* C = reinterpret_cast<uint64_t*>(smem + L.off_C);
  uint32_t* w = reinterpret_cast<uint32_t*>(smem + L.off_w);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + L.off_cnt);
  int32_t* uidx = reinterpret_cast<int32_t*>(smem + L.off_uidx);
  float* ucoef = reinterpret_cast<float*>(smem + L.off_ucoef);
  float* misc_f = reinterpret_cast<float*>(smem + L.off_misc);           // [4]
  uint64_t* misc_u64 = reinterpret_cast<uint64_t*>(smem + L.off_misc + 16);  // [4]
  int32_t* misc_i = reinterpret_cast<int32_t*>(smem + L.off_misc + 48);  // [4]

  // ---- 2. fixed-point sampling weights
  const T* xrow = static_cast<const T*>(p.X) + tok * d_in;
  float lmax = 0.f;
  for (int i = tid; i < d_in; i += kThreads) {
    const float v = __fmul_rn(fabsf(load_f32(xrow, i)), p.rownorm[i]);
    w[i] = __float_as_uint(v);
    cnt[i] = 0u;
    lmax = fmaxf(lmax, v);
  }
  lmax = wave_max(lmax);
  if (lane == 0) misc_f[wave] = lmax;
  __syncthreads();
  const float vmax = fmaxf(fmaxf(misc_f[0], misc_f[1]), fmaxf(misc_f[2], misc_f[3]));
  if (!(vmax > 0.f) || !(vmax <= 3.40282347e38f)) {  // x_j = 0 (or non-finite): H~[j] = 0
    write_zero_row<BF>(p, tok, tid);
    return;
  }
  int e;
  (void)frexpf(vmax, &e);  // vmax = f 2^e, f in [0.5, 1)
  const int shift = 32 - e;

  // contiguous chunk of rows per thread for the scans
  const int per = (d_in + kThreads - 1) / kThreads;
  const int i0 = min(tid * per, d_in), i1 = min(i0 + per, d_in);
  for (int i = i0; i < i1; ++i) w[i] = (uint32_t)ldexpf(__uint_as_float(w[i]), shift);
  uint64_t part = 0;
  for (int i = i0; i < i1; ++i) part += w[i];
  uint64_t T_total;
  uint64_t run = block_exclusive_scan<uint64_t>(part, misc_u64, &T_total, lane, wave);
  for (int i = i0; i < i1; ++i) {
    run += w[i];
    C[i] = run;
  }
  __syncthreads();
  const uint64_t Tw = C[d_in - 1];

  // ---- 3. draws
  for (int k = tid; k < r; k += kThreads) {
    const u32x4 o = philox4x32_10(u32x4{(uint32_t)k, (uint32_t)j, (uint32_t)b, 0u}, p.seed_lo, p.seed_hi);
    const uint64_t u = (uint64_t)o.x | ((uint64_t)o.y << 32);
    const uint64_t t = __umul64hi(u, Tw);  // in [0, T)
    int lo = 0, hi = d_in - 1;             // C[d_in-1] = T > t, so the answer is in range
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (C[mid] > t) hi = mid;
      else lo = mid + 1;
    }
    atomicAdd(cnt + lo, 1u);
    const int64_t o2 = tok * d_in + k;
    if (p.idx_out) p.idx_out[o2] = lo;
    if (p.coef_out)
      p.coef_out[o2] = (float)(((double)load_f32(xrow, lo) * (double)Tw) / ((double)r * (double)w[lo]));
  }
  __syncthreads();

  // ---- 4. merge duplicates, compact in ascending row order
  int nloc = 0;
  for (int i = i0; i < i1; ++i) nloc += cnt[i] != 0u;
  int U;
  int pos = block_exclusive_scan<int32_t>(nloc, misc_i, &U, lane, wave);
  for (int i = i0; i < i1; ++i) {
    const uint32_t c = cnt[i];
    if (c) {
      uidx[pos] = i;
      ucoef[pos] = (float)(((double)c * (double)load_f32(xrow, i) * (double)Tw) / ((double)r * (double)w[i]));
      ++pos;
    }
  }
  __syncthreads();

  // ---- 5. gather-scale-accumulate (lane owns columns (v*64 + lane)*4 .. +3)
  float4 acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = make_float4(0.f, 0.f, 0.f, 0.f);
  const T* W = static_cast<const T*>(p.W);
  int qi = wave;
  for (; qi + 3 * kWaves < U; qi += 4 * kWaves) {
    int rows[4];
    float cs[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      rows[u] = uidx[qi + u * kWaves];
      cs[u] = ucoef[qi + u * kWaves];
    }
    float4 wv[4][NV];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < NV; ++v) wv[u][v] = load4_f32(W + (int64_t)rows[u] * d_out + (v * kWave + lane) * 4);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        acc[v].x = fmaf(cs[u], wv[u][v].x, acc[v].x);
        acc[v].y = fmaf(cs[u], wv[u][v].y, acc[v].y);
        acc[v].z = fmaf(cs[u], wv[u][v].z, acc[v].z);
        acc[v].w = fmaf(cs[u], wv[u][v].w, acc[v].w);
      }
  }
  for (; qi < U; qi += kWaves) {
    const int row = uidx[qi];
    const float c = ucoef[qi];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const float4 x = load4_f32(W + (int64_t)row * d_out + (v * kWave + lane) * 4);
      acc[v].x = fmaf(c, x.x, acc[v].x);
      acc[v].y = fmaf(c, x.y, acc[v].y);
      acc[v].z = fmaf(c, x.z, acc[v].z);
      acc[v].w = fmaf(c, x.w, acc[v].w);
    }
  }

  // partial rows of the four waves, summed in wave order
  float* red = reinterpret_cast<float*>(smem);  // [4][d_out], aliases C / w / cnt (no longer read)
#pragma unroll
  for (int v = 0; v < NV; ++v) *reinterpret_cast<float4*>(red + wave * d_out + (v * kWave + lane) * 4) = acc[v];
  __syncthreads();
  for (int c = 4 * tid; c < d_out; c += 4 * kThreads) {
    const float4 a0 = *reinterpret_cast<const float4*>(red + c);
    const float4 a1 = *reinterpret_cast<const float4*>(red + d_out + c);
    const float4 a2 = *reinterpret_cast<const float4*>(red + 2 * d_out + c);
    const float4 a3 = *reinterpret_cast<const float4*>(red + 3 * d_out + c);
    const float4 s = make_float4(((a0.x + a1.x) + a2.x) + a3.x, ((a0.y + a1.y) + a2.y) + a3.y,
                                 ((a0.z + a1.z) + a2.z) + a3.z, ((a0.w + a1.w) + a2.w) + a3.w);
    write_row<BF>(p, tok, s, c);
  }
}

// rho_i = float32(sqrt(sum_c W[i, c]^2)), float64 running sum in column order. One wave
// per 64 rows; 64x64 tiles go through LDS so global reads are coalesced.
template <int BF>
__global__ __launch_bounds__(64) void k_rownorm(const void* Wp, int d_in, int d_out, float* rownorm) {
  using T = typename Elem<BF>::T;
  __shared__ double tile[64][65];
  const T* W = static_cast<const T*>(Wp);
  const int r0 = blockIdx.x * 64, lane = threadIdx.x;
  double s = 0.0;
  for (int c0 = 0; c0 < d_out; c0 += 64) {
    for (int rr = 0; rr < 64; ++rr) {
      const int row = r0 + rr, c = c0 + lane;
      tile[rr][lane] = (row < d_in && c < d_out) ? (double)load_f32(W, (int64_t)row * d_out + c) : 0.0;
    }
    __syncthreads();
    const int cend = min(64, d_out - c0);
    for (int cc = 0; cc < cend; ++cc) {
      const double v = tile[lane][cc];
      s = __dadd_rn(s, __dmul_rn(v, v));  // v*v is exact in float64
    }
    __syncthreads();
  }
  if (r0 + lane < d_in) rownorm[r0 + lane] = (float)sqrt(s);
}

template <int BF>
hipError_t launch_encode_dt(const FwdParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)p.B * p.n));
  const size_t lds = encode_lds_layout(p.d_in, p.d_out).total;
  switch (p.d_out / 256) {
    case 1: hipLaunchKernelGGL((k_encode<BF, 1>), grid, dim3(kThreads), lds, s, p); break;
    case 2: hipLaunchKernelGGL((k_encode<BF, 2>), grid, dim3(kThreads), lds, s, p); break;
    case 3: hipLaunchKernelGGL((k_encode<BF, 3>), grid, dim3(kThreads), lds, s, p); break;
    case 4: hipLaunchKernelGGL((k_encode<BF, 4>), grid, dim3(kThreads), lds, s, p); break;
    case 5: hipLaunchKernelGGL((k_encode<BF, 5>), grid, dim3(kThreads), lds, s, p); break;
    case 6: hipLaunchKernelGGL((k_encode<BF, 6>), grid, dim3(kThreads), lds, s, p); break;
    case 7: hipLaunchKernelGGL((k_encode<BF, 7>), grid, dim3(kThreads), lds, s, p); break;
    case 8: hipLaunchKernelGGL((k_encode<BF, 8>), grid, dim3(kThreads), lds, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

size_t encode_lds_bytes(int d_in, int d_out) { return (size_t)encode_lds_layout(d_in, d_out).total; }

hipError_t launch_encode(const FwdParams& p, hipStream_t s) {
  return p.bf16 ? launch_encode_dt<1>(p, s) : launch_encode_dt<0>(p, s);
}

hipError_t launch_rownorm(const void* W, int bf16, int d_in, int d_out, float* rownorm, hipStream_t s) {
  const dim3 grid((d_in + 63) / 64);
  if (bf16) hipLaunchKernelGGL(k_rownorm<1>, grid, dim3(64), 0, s, W, d_in, d_out, rownorm);
  else hipLaunchKernelGGL(k_rownorm<0>, grid, dim3(64), 0, s, W, d_in, d_out, rownorm);
  return hipGetLastError();
}

}  // namespace mca
