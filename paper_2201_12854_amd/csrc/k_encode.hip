// Sampled value encoding of the MCA forward pass on gfx950.
//
// One block (NW waves) per token j of batch row b:
//   1. column max m_j = max over the per-(head, query tile) partials written by the score
//      pass, and the sample count of Eq. 9 (Sec. "Determining Sample Size from
//      Attention") in float64: t = (len_b * m_j) / alpha, r_j = ceil(t * t) clamped to
//      [1, d_in]; padded keys get 0; r_j = d_in leaves the token to the exact MFMA path.
//   2. sampling weights of Eq. 4 for the product x_j W_v: v_i = |x_ji| * rho_i in one
//      float32 multiply, quantised to 32-bit fixed point aligned to the largest v_i,
//      w_i = floor(v_i 2^(32-e)); inclusive prefix sums C (uint64) in LDS.
//   3. r_j i.i.d. draws with replacement (Eq. 2): Philox4x32-10 with counter
//      (k, j, b, 0), u = o0 | o1 << 32, t = floor(u T / 2^64), s_k = min{i : C_i > t}
//      by binary search in LDS. Draws are counted per row with LDS integer atomics
//      (exact, order-free).
//   4. duplicates merged: coefficient of row i = count_i x_ji T / (r_j w_i) (float64,
//      rounded once), rows compacted in ascending order.
//   5. gather-scale-accumulate: the waves split the distinct rows of W_v; each half-wave
//      streams one row with 16-byte loads (several rows in flight), accumulating in
//      float32; the partial rows are summed in a fixed order through LDS.
// The loads of m, x and rho are issued together at block start. Everything is
// deterministic: the same inputs and seed give bitwise-equal output.
//
// Also here: the one-time weight preparation (Sec. "Formulation of Sampling
// Probability": the per-row statistic of W is computed once and cached), row norms and
// a zero-padded transposed copy of W_v for the MFMA path.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

constexpr int kMaxDin = 2048;

struct EncodeLds {
  int off_C, off_cnt, off_uidx, off_ucoef, off_misc, total;
};

__host__ __device__ inline int round_up(int v, int a) { return (v + a - 1) / a * a; }

__host__ __device__ inline EncodeLds encode_lds_layout(int d_in, int d_out, int nw) {
  EncodeLds l;
  l.off_C = 0;           // uint64 [d_in]
  l.off_cnt = 8 * d_in;  // uint32 [d_in]
  // the partial-row reduction buffer float [nw][d_out] aliases C and cnt
  const int a = 12 * d_in, bsz = 4 * nw * d_out;
  const int region0 = round_up(a > bsz ? a : bsz, 16);
  l.off_uidx = region0;              // int32 [d_in]
  l.off_ucoef = region0 + 4 * d_in;  // float [d_in]
  l.off_misc = round_up(region0 + 8 * d_in, 16);
  l.total = l.off_misc + 32 * nw;  // per wave: float max, float m, uint64 scan, int32 scan
  return l;
}

// 16-byte chunk of a W_v row: 8 bf16 or 4 float32 columns.
template <int BF> struct Row16;
template <> struct Row16<1> {
  static constexpr int kElems = 8;
  static __device__ __forceinline__ float at(const uint4& v, int e) {
    const uint32_t w = e < 2 ? v.x : e < 4 ? v.y : e < 6 ? v.z : v.w;
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  }
};
template <> struct Row16<0> {
  static constexpr int kElems = 4;
  static __device__ __forceinline__ float at(const uint4& v, int e) {
    return __uint_as_float(e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w);
  }
};

// Writes 4 consecutive H~ columns (and the float32 export).
template <int BF>
__device__ __forceinline__ void write_row4(const FwdParams& p, int64_t off, float4 v) {
  if constexpr (BF) {
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.Henc) + off) =
        make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(p.Henc) + off) = v;
  }
  if (p.enc_out) *reinterpret_cast<float4*>(p.enc_out + off) = v;
}

template <int BF, int NT>
__device__ void write_zero_row(const FwdParams& p, int64_t tok, int tid) {
  for (int c = 4 * tid; c < p.d_out; c += 4 * NT) write_row4<BF>(p, tok * p.d_out + c, make_float4(0.f, 0.f, 0.f, 0.f));
}

// Exclusive prefix (thread order) of a per-thread value and the block total; `scratch`
// holds NW values. Contains one barrier.
template <int NW, typename U>
__device__ __forceinline__ U block_exclusive_scan(U v, U* scratch, U* total, int lane, int wave) {
  U incl = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const U y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) scratch[wave] = incl;
  lds_barrier();
  U base = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if (w < wave) base += scratch[w];
    all += scratch[w];
  }
  *total = all;
  return base + incl - v;
}

template <int BF, int NV, int NW>
__global__ __launch_bounds__(64 * NW) void k_encode(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int NT = 64 * NW;
  constexpr int MAXPER = (kMaxDin + NT - 1) / NT;
  extern __shared__ __align__(16) unsigned char smem[];
  const int d_in = p.d_in, d_out = p.d_out, n = p.n;
  const int64_t tok = blockIdx.x;
  const int b = (int)(tok / n), j = (int)(tok - (int64_t)b * n);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  const EncodeLds L = encode_lds_layout(d_in, d_out, NW);
  uint64_t* C = reinterpret_cast<uint64_t*>(smem + L.off_C);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + L.off_cnt);
  int32_t* uidx = reinterpret_cast<int32_t*>(smem + L.off_uidx);
  float* ucoef = reinterpret_cast<float*>(smem + L.off_ucoef);
  float* misc_vmax = reinterpret_cast<float*>(smem + L.off_misc);
  float* misc_m = misc_vmax + NW;
  uint64_t* misc_u64 = reinterpret_cast<uint64_t*>(smem + L.off_misc + 8 * NW);
  int32_t* misc_i = reinterpret_cast<int32_t*>(smem + L.off_misc + 16 * NW);

  // ---- independent loads first: length, column-max partials, x and rho of this thread's
  // contiguous chunk of rows
  int len = p.seq_lens ? p.seq_lens[b] : n;
  len = min(max(len, 1), n);
  const int rin = p.r_in ? p.r_in[tok] : 0;
  const float* part = p.colmax_part + tok * p.nparts;
  float mloc = 0.f;
  for (int t = tid; t < p.nparts; t += NT) mloc = fmaxf(mloc, part[t]);
  const int per = (d_in + NT - 1) / NT;
  const int i0 = min(tid * per, d_in), i1 = min(i0 + per, d_in);
  const T* xrow = static_cast<const T*>(p.X) + tok * d_in;
  float xv[MAXPER], vv[MAXPER];
  float lmax = 0.f;
#pragma unroll
  for (int k = 0; k < MAXPER; ++k) {
    xv[k] = 0.f;
    vv[k] = 0.f;
    if (k < i1 - i0) {
      xv[k] = load_f32(xrow, i0 + k);
      vv[k] = __fmul_rn(fabsf(xv[k]), p.rownorm[i0 + k]);
      lmax = fmaxf(lmax, vv[k]);
      cnt[i0 + k] = 0u;
    }
  }
  mloc = wave_max(mloc);
  lmax = wave_max(lmax);
  if (lane == 0) {
    misc_m[wave] = mloc;
    misc_vmax[wave] = lmax;
  }
  lds_barrier();
  float m = misc_m[0], vmax = misc_vmax[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    m = fmaxf(m, misc_m[w]);
    vmax = fmaxf(vmax, misc_vmax[w]);
  }

  // ---- 1. sample count (Eq. 9)
  int r;
  if (j >= len) {
    r = 0;
    m = 0.f;
  } else if (p.r_in) {
    r = min(max(rin, 0), d_in);
  } else {
    const double t = ((double)len * (double)m) / p.alpha;
    const double tt = t * t;
    r = (tt >= (double)d_in) ? d_in : max((int)ceil(tt), 1);
  }
  if (tid == 0) {
    p.r[tok] = r;
    if (p.colmax_out) p.colmax_out[tok] = m;
  }
  if (r >= d_in) return;  // saturated: exact encoding by the MFMA path
  if (r == 0 || !(vmax > 0.f) || !(vmax <= 3.40282347e38f)) {  // padded, x_j = 0 or non-finite
    write_zero_row<BF, NT>(p, tok, tid);
    return;
  }

  // ---- 2. fixed-point weights and their prefix sums
  int e;
  (void)frexpf(vmax, &e);  // vmax = f 2^e, f in [0.5, 1)
  const int shift = 32 - e;
  uint32_t wv[MAXPER];
  uint64_t part_sum = 0;
#pragma unroll
  for (int k = 0; k < MAXPER; ++k) {
    wv[k] = (k < i1 - i0) ? (uint32_t)ldexpf(vv[k], shift) : 0u;
    part_sum += wv[k];
  }
  uint64_t T_total;
  uint64_t run = block_exclusive_scan<NW, uint64_t>(part_sum, misc_u64, &T_total, lane, wave);
#pragma unroll
  for (int k = 0; k < MAXPER; ++k) {
    if (k < i1 - i0) {
      run += wv[k];
      C[i0 + k] = run;
    }
  }
  lds_barrier();
  const uint64_t Tw = T_total;  // = C[d_in - 1]

  // ---- 3. draws
  for (int k = tid; k < r; k += NT) {
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
    if (p.coef_out) {
      const uint64_t ws = C[lo] - (lo > 0 ? C[lo - 1] : 0ull);
      p.coef_out[o2] = (float)(((double)load_f32(xrow, lo) * (double)Tw) / ((double)r * (double)ws));
    }
  }
  lds_barrier();

  // ---- 4. merge duplicates, compact in ascending row order
  int nloc = 0;
#pragma unroll
  for (int k = 0; k < MAXPER; ++k)
    if (k < i1 - i0) nloc += cnt[i0 + k] != 0u;
  int U;
  int pos = block_exclusive_scan<NW, int32_t>(nloc, misc_i, &U, lane, wave);
#pragma unroll
  for (int k = 0; k < MAXPER; ++k) {
    if (k < i1 - i0) {
      const uint32_t c = cnt[i0 + k];
      if (c) {
        uidx[pos] = i0 + k;
        ucoef[pos] = (float)(((double)c * (double)xv[k] * (double)Tw) / ((double)r * (double)wv[k]));
        ++pos;
      }
    }
  }
  lds_barrier();

  // ---- 5. gather-scale-accumulate. Each half of a wave streams its own row with 16-byte
  // loads (lane hl = lane % 32 owns columns v * 32E + hl * E .. +E-1, E = 8 bf16 / 4 f32
  // per chunk); the two halves take alternate entries of the wave's share of the list,
  // GU rows in flight each, and are added together at the end.
  using RC = Row16<BF>;
  constexpr int E = RC::kElems;
  constexpr int VPL = NV * 8 / E;  // 16-byte chunks per lane per row
  constexpr int GU = VPL <= 3 ? 4 : (VPL <= 6 ? 2 : 1);
  const int half = lane >> 5, hl = lane & 31;
  float acc[VPL * E];
#pragma unroll
  for (int k = 0; k < VPL * E; ++k) acc[k] = 0.f;
  const T* W = static_cast<const T*>(p.W) + hl * E;
  const int step = 2 * NW;
  int q = 2 * wave + half;
  for (; q + (GU - 1) * step < U; q += GU * step) {
    uint4 raw[GU][VPL];
    float cs[GU];
#pragma unroll
    for (int u = 0; u < GU; ++u) {
      const int row = uidx[q + u * step];
      cs[u] = ucoef[q + u * step];
#pragma unroll
      for (int v = 0; v < VPL; ++v) raw[u][v] = *reinterpret_cast<const uint4*>(W + (int64_t)row * d_out + v * 32 * E);
    }
#pragma unroll
    for (int u = 0; u < GU; ++u)
#pragma unroll
      for (int v = 0; v < VPL; ++v)
#pragma unroll
        for (int e = 0; e < E; ++e) acc[v * E + e] = fmaf(cs[u], RC::at(raw[u][v], e), acc[v * E + e]);
  }
  for (; q < U; q += step) {
    const int row = uidx[q];
    const float c = ucoef[q];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const uint4 raw = *reinterpret_cast<const uint4*>(W + (int64_t)row * d_out + v * 32 * E);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[v * E + e] = fmaf(c, RC::at(raw, e), acc[v * E + e]);
    }
  }
#pragma unroll
  for (int k = 0; k < VPL * E; ++k) acc[k] += __shfl_xor(acc[k], 32, kWave);

  // partial rows of the waves, summed in wave order (aliases C / cnt, no longer read)
  float* red = reinterpret_cast<float*>(smem);
  if (half == 0) {
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int e = 0; e < E; e += 4)
        *reinterpret_cast<float4*>(red + wave * d_out + v * 32 * E + hl * E + e) =
            make_float4(acc[v * E + e], acc[v * E + e + 1], acc[v * E + e + 2], acc[v * E + e + 3]);
  }
  lds_barrier();
  for (int c = 4 * tid; c < d_out; c += 4 * NT) {
    float4 s = *reinterpret_cast<const float4*>(red + c);
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      const float4 a = *reinterpret_cast<const float4*>(red + w * d_out + c);
      s.x += a.x;
      s.y += a.y;
      s.z += a.z;
      s.w += a.w;
    }
    write_row4<BF>(p, tok * d_out + c, s);
  }
}

// ------------------------------------------------------------------ weight preparation
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
    lds_barrier();
    const int cend = min(64, d_out - c0);
    for (int cc = 0; cc < cend; ++cc) {
      const double v = tile[lane][cc];
      s = __dadd_rn(s, __dmul_rn(v, v));  // v*v is exact in float64
    }
    lds_barrier();
  }
  if (r0 + lane < d_in) rownorm[r0 + lane] = (float)sqrt(s);
}

// Wt[c][i] = W[i][c] for i < d_in, 0 for d_in <= i < din_pad (64x64 tiles through LDS).
template <int BF>
__global__ __launch_bounds__(256) void k_transpose_pad(const void* Wp, int d_in, int d_out, int din_pad, void* Wtp) {
  using T = typename Elem<BF>::T;
  __shared__ T tile[64][65];
  const T* W = static_cast<const T*>(Wp);
  T* Wt = static_cast<T*>(Wtp);
  const int i0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int rr = ty; rr < 64; rr += 4) {
    const int i = i0 + rr, c = c0 + tx;
    tile[rr][tx] = (i < d_in && c < d_out) ? W[(int64_t)i * d_out + c] : T(0);
  }
  lds_barrier();
  for (int cc = ty; cc < 64; cc += 4) {
    const int c = c0 + cc, i = i0 + tx;
    if (c < d_out && i < din_pad) Wt[(int64_t)c * din_pad + i] = tile[tx][cc];
  }
}

template <int BF, int NW>
hipError_t launch_encode_nw(const FwdParams& p, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)p.B * p.n));
  const size_t lds = encode_lds_layout(p.d_in, p.d_out, NW).total;
  switch (p.d_out / 256) {
    case 1: hipLaunchKernelGGL((k_encode<BF, 1, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 2: hipLaunchKernelGGL((k_encode<BF, 2, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 3: hipLaunchKernelGGL((k_encode<BF, 3, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 4: hipLaunchKernelGGL((k_encode<BF, 4, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 5: hipLaunchKernelGGL((k_encode<BF, 5, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 6: hipLaunchKernelGGL((k_encode<BF, 6, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 7: hipLaunchKernelGGL((k_encode<BF, 7, NW>), grid, dim3(64 * NW), lds, s, p); break;
    case 8: hipLaunchKernelGGL((k_encode<BF, 8, NW>), grid, dim3(64 * NW), lds, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

#ifndef MCA_ENCODE_WAVES
#define MCA_ENCODE_WAVES 4
#endif

}  // namespace

hipError_t launch_encode(const FwdParams& p, hipStream_t s) {
  return p.bf16 ? launch_encode_nw<1, MCA_ENCODE_WAVES>(p, s) : launch_encode_nw<0, MCA_ENCODE_WAVES>(p, s);
}

hipError_t launch_prepare(const void* W, int bf16, int d_in, int d_out, void* prepared, hipStream_t s) {
  float* rownorm = static_cast<float*>(prepared);
  void* Wt = static_cast<char*>(prepared) + prepared_wt_offset(d_in);
  const int din_pad = (int)prepared_din_pad(d_in);
  const dim3 g1((d_in + 63) / 64);
  const dim3 g2((din_pad + 63) / 64, (d_out + 63) / 64);
  if (bf16) {
    hipLaunchKernelGGL(k_rownorm<1>, g1, dim3(64), 0, s, W, d_in, d_out, rownorm);
    hipLaunchKernelGGL(k_transpose_pad<1>, g2, dim3(256), 0, s, W, d_in, d_out, din_pad, Wt);
  } else {
    hipLaunchKernelGGL(k_rownorm<0>, g1, dim3(64), 0, s, W, d_in, d_out, rownorm);
    hipLaunchKernelGGL(k_transpose_pad<0>, g2, dim3(256), 0, s, W, d_in, d_out, din_pad, Wt);
  }
  return hipGetLastError();
}

}  // namespace mca
