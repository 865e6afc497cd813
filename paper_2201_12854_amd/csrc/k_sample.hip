// Sampler of the MCA forward pass on gfx950: one wavefront per token j of batch row b.
//
//   1. column max m_j = max over the per-(head, query tile) partials written by the score
//      pass, and the sample count of Eq. 9 (Sec. "Determining Sample Size from
//      Attention") in float64: t = (len_b * m_j) / alpha, r_j = ceil(t * t) clamped to
//      [1, d_in]; padded keys get 0. r_j = d_in marks a saturated token, encoded exactly
//      by the gather kernel's MFMA path (cost of d_in samples, no error).
//   2. sampling weights of Eq. 4 for the product x_j W_v: v_i = |x_ji| * rho_i in one
//      float32 multiply, quantised to 32-bit fixed point aligned to the largest v_i,
//      w_i = floor(v_i 2^(32-e)); inclusive prefix sums C (uint64) by a wavefront scan
//      (each lane owns a contiguous run of rows), stored in the wave's part of the LDS.
//      In the paper's input-independent mode (Eq. 6, p_i ~ rho_i^2) the prefix sums are
//      the same for every token: they come precomputed with the prepared weights and are
//      copied into LDS once per block.
//   3. r_j i.i.d. draws with replacement (Eq. 2): Philox4x32-10 with counter (k, j, b, 0),
//      u = o0 | o1 << 32, t = floor(u T / 2^64), s_k = min{i : C_i > t} by binary search
//      in LDS; draws are counted per row with LDS integer atomics (exact, order-free).
//   4. duplicates merged: coefficient of row i = count_i x_ji T / (r_j w_i) (float64,
//      rounded once); the distinct rows with their coefficients form the token's list
//      (rows as byte offsets into the gather kernel's LDS slice): even rows first, then
//      odd rows, each part ascending and padded to an even length with a zero row of its
//      parity. ucount gets (even part length << 16) | total length, 0 for tokens without
//      a list.
// A wave works on its own token and its own LDS region only (under Eq. 6 the block first
// shares the copied table behind one barrier): no global atomics (on a multi-die GPU,
// device-scope atomics on a few hot counters serialise). Everything it writes is
// deterministic.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

constexpr int kWaves = 4;  // tokens per block

// LDS of one wave: C uint64 [d_in], then cnt uint32 [d_in].
__host__ __device__ inline int sample_lds_per_wave(int d_in) { return (12 * d_in + 15) / 16 * 16; }

// Orders LDS accesses of different lanes of one wavefront: the hardware executes a wave's
// LDS instructions in issue order, so only compiler reordering has to be prevented.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

template <typename U>
__device__ __forceinline__ U wave_inclusive_scan(U v, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const U y = __shfl_up(v, off, kWave);
    if (lane >= off) v += y;
  }
  return v;
}

template <int BF>
__device__ __forceinline__ void write_zero4(const FwdParams& p, int64_t off) {
  if constexpr (BF) *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.Henc) + off) = make_uint2(0u, 0u);
  else *reinterpret_cast<float4*>(static_cast<float*>(p.Henc) + off) = make_float4(0.f, 0.f, 0.f, 0.f);
  if (p.enc_out) *reinterpret_cast<float4*>(p.enc_out + off) = make_float4(0.f, 0.f, 0.f, 0.f);
}

// W draws of one lane, k = k0 + 64 u (u < W), searched together so that their LDS reads
// overlap. The search runs a fixed number of halvings (ceil(log2 d_in)) without branches;
// once lo == hi it stays put, since C[lo] > t there.
template <int W>
__device__ __forceinline__ void draw_batch(const FwdParams& p, const uint64_t* C, uint32_t* cnt, const void* xrow,
                                           int k0, int r, int j, int b, int64_t tok, uint64_t Tw, int nsteps) {
  uint64_t t[W];
  int lo[W], hi[W];
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const int k = k0 + u * kWave;
    const u32x4 o = philox4x32_10(u32x4{(uint32_t)k, (uint32_t)j, (uint32_t)b, 0u}, p.seed_lo, p.seed_hi);
    t[u] = __umul64hi((uint64_t)o.x | ((uint64_t)o.y << 32), Tw);  // in [0, T)
    lo[u] = 0;
    hi[u] = p.d_in - 1;  // C[d_in-1] = T > t, so the answer is in range
  }
  for (int st = 0; st < nsteps; ++st) {
#pragma unroll
    for (int u = 0; u < W; ++u) {
      const int mid = (lo[u] + hi[u]) >> 1;
      const bool right = C[mid] <= t[u];
      lo[u] = right ? mid + 1 : lo[u];
      hi[u] = right ? hi[u] : mid;
    }
  }
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const int k = k0 + u * kWave;
    if (k < r) {
      atomicAdd(cnt + lo[u], 1u);
      const int64_t o2 = tok * p.d_in + k;
      if (p.idx_out) p.idx_out[o2] = lo[u];
      if (p.coef_out) {
        const uint64_t ws = C[lo[u]] - (lo[u] > 0 ? C[lo[u] - 1] : 0ull);
        const double xs = p.bf16 ? (double)load_f32(static_cast<const uint16_t*>(xrow), lo[u])
                                 : (double)load_f32(static_cast<const float*>(xrow), lo[u]);
        p.coef_out[o2] = (float)((xs * (double)Tw) / ((double)r * (double)ws));
      }
    }
  }
}

// PER: upper bound of the rows one lane owns, ceil(d_in / 64) <= PER.
// LDS of a block. Per-token weights (Eq. 4): per wave C uint64 [d_in] then cnt uint32
// [d_in]. Shared table (Eq. 6): C uint64 [d_in] once per block, then cnt per wave.
__host__ __device__ inline int round16(int v) { return (v + 15) / 16 * 16; }
__host__ __device__ inline int sample_lds_bytes(int d_in, bool table) {
  return table ? round16(8 * d_in) + kWaves * round16(4 * d_in) : kWaves * sample_lds_per_wave(d_in);
}

// PER: upper bound of the rows one lane owns, ceil(d_in / 64) <= PER. TABLE: the
// input-independent probability of Eq. 6, whose prefix sums come from the prepared
// weights (copied into LDS once per block and shared by its tokens); otherwise the
// per-token probability of Eq. 4, quantised and scanned per token.
template <int BF, int PER, bool TABLE>
__global__ __launch_bounds__(64 * kWaves) void k_sample(FwdParams p) {
  using T = typename Elem<BF>::T;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ntok = (int64_t)p.B * p.n;
  const int64_t tok = (int64_t)blockIdx.x * kWaves + wave;
  const int d_in = p.d_in, n = p.n;
  uint64_t* C;
  uint32_t* cnt;
  if constexpr (TABLE) {
    C = reinterpret_cast<uint64_t*>(smem);
    cnt = reinterpret_cast<uint32_t*>(smem + round16(8 * d_in) + wave * round16(4 * d_in));
    for (int i = threadIdx.x; i < d_in; i += 64 * kWaves) C[i] = p.wtable[i];
    __syncthreads();  // the only block barrier; waves without a token return after it
  } else {
    unsigned char* wl = smem + wave * sample_lds_per_wave(d_in);
    C = reinterpret_cast<uint64_t*>(wl);
    cnt = reinterpret_cast<uint32_t*>(wl + 8 * d_in);
  }
  if (tok >= ntok) return;  // whole waves only; no block barrier follows
  const int b = (int)(tok / n), j = (int)(tok - (int64_t)b * n);

  // ---- independent loads first: length, column-max partials, x (and rho under Eq. 4) of
  // this lane's contiguous run of rows [i0, i0 + nrows)
  int len = p.seq_lens ? p.seq_lens[b] : n;
  len = min(max(len, 1), n);
  const int rin = p.r_in ? p.r_in[tok] : 0;
  const float* part = p.colmax_part + tok * p.nparts;
  float m = 0.f;
  for (int t = lane; t < p.nparts; t += kWave) m = fmaxf(m, part[t]);
  const int per = (d_in + kWave - 1) / kWave;
  const int i0 = min(lane * per, d_in);
  const int nrows = min(per, d_in - i0);
  const T* xrow = static_cast<const T*>(p.X) + tok * d_in;
  // full: d_in = 64 PER, every lane owns exactly PER rows and its runs of x, rho, C and
  // cnt are 16-byte aligned (i0 = PER lane), so they move as 16-byte vectors
  const bool full = d_in == kWave * PER;
  float xv[PER], vv[PER];
  float lmax = 0.f;
  if (full) {
#pragma unroll
    for (int k = 0; k < PER; k += 4) {
      const float4 xs = load4_f32(xrow + i0 + k);
      xv[k] = xs.x; xv[k + 1] = xs.y; xv[k + 2] = xs.z; xv[k + 3] = xs.w;
      if constexpr (!TABLE) {
        const float4 rs = *reinterpret_cast<const float4*>(p.rownorm + i0 + k);
        vv[k] = __fmul_rn(fabsf(xs.x), rs.x);
        vv[k + 1] = __fmul_rn(fabsf(xs.y), rs.y);
        vv[k + 2] = __fmul_rn(fabsf(xs.z), rs.z);
        vv[k + 3] = __fmul_rn(fabsf(xs.w), rs.w);
      }
    }
    if constexpr (!TABLE) {
#pragma unroll
      for (int k = 0; k < PER; ++k) lmax = fmaxf(lmax, vv[k]);
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      xv[k] = 0.f;
      vv[k] = 0.f;
      if (k < nrows) {
        xv[k] = load_f32(xrow, i0 + k);
        if constexpr (!TABLE) {
          vv[k] = __fmul_rn(fabsf(xv[k]), p.rownorm[i0 + k]);
          lmax = fmaxf(lmax, vv[k]);
        }
      }
    }
  }
  m = wave_max(m);

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
  if (lane == 0) {
    p.r[tok] = r;
    if (p.colmax_out) p.colmax_out[tok] = m;
  }
  if (r >= d_in) {  // saturated: exact encoding on the MFMA path of the gather kernel
    if (lane == 0) p.ucount[tok] = 0;
    return;
  }

  // ---- 2. the distribution: per-token fixed-point weights and their prefix sums (Eq. 4),
  // or the shared table (Eq. 6). No distribution (x_j = 0 under Eq. 4, W_v = 0 under
  // Eq. 6, non-finite weights) or a padded key: H~[j] = 0.
  uint32_t wv[PER];
  uint64_t Tw;
  bool none;
  if constexpr (TABLE) {
    Tw = C[d_in - 1];
    none = Tw == 0;
  } else {
    const float vmax = wave_max(lmax);
    none = !(vmax > 0.f) || !(vmax <= 3.40282347e38f);
    Tw = 0;
    if (!none) {
      int e;
      (void)frexpf(vmax, &e);  // vmax = f 2^e, f in [0.5, 1)
      const int shift = 32 - e;
      uint64_t lsum = 0;
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        wv[k] = (k < nrows) ? (uint32_t)ldexpf(vv[k], shift) : 0u;
        lsum += wv[k];
      }
      const uint64_t incl = wave_inclusive_scan<uint64_t>(lsum, lane);
      Tw = __shfl(incl, kWave - 1, kWave);  // = C[d_in - 1]
      uint64_t run = incl - lsum;
      if (full) {
#pragma unroll
        for (int k = 0; k < PER; k += 2) {
          const uint64_t c0 = run + wv[k], c1 = c0 + wv[k + 1];
          run = c1;
          *reinterpret_cast<uint4*>(C + i0 + k) =
              make_uint4((uint32_t)c0, (uint32_t)(c0 >> 32), (uint32_t)c1, (uint32_t)(c1 >> 32));
        }
      } else {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          if (k < nrows) {
            run += wv[k];
            C[i0 + k] = run;
          }
        }
      }
    }
  }
  if (r == 0 || none) {
    if (lane == 0) p.ucount[tok] = 0;
    for (int c = 4 * lane; c < p.d_out; c += 4 * kWave) write_zero4<BF>(p, tok * p.d_out + c);
    return;
  }
  if (full) {
#pragma unroll
    for (int k = 0; k < PER; k += 4) *reinterpret_cast<uint4*>(cnt + i0 + k) = make_uint4(0u, 0u, 0u, 0u);
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k)
      if (k < nrows) cnt[i0 + k] = 0u;
  }
  wave_lds_sync();

  // ---- 3. draws: ceil(r / 64) per lane, in batches of up to 4 searched together
  const int nsteps = 32 - __clz(max(d_in - 1, 1));
  const int nper = (r + kWave - 1) / kWave;
  for (int u0 = 0; u0 < nper; u0 += 4) {
    const int k0 = lane + u0 * kWave;
    const int w = min(4, nper - u0);
    if (w == 4) draw_batch<4>(p, C, cnt, xrow, k0, r, j, b, tok, Tw, nsteps);
    else if (w == 3) draw_batch<3>(p, C, cnt, xrow, k0, r, j, b, tok, Tw, nsteps);
    else if (w == 2) draw_batch<2>(p, C, cnt, xrow, k0, r, j, b, tok, Tw, nsteps);
    else draw_batch<1>(p, C, cnt, xrow, k0, r, j, b, tok, Tw, nsteps);
  }
  wave_lds_sync();

  // ---- 4. merge duplicates into the token's list, ascending row order
  uint32_t cv[PER];
  if (full) {
#pragma unroll
    for (int k = 0; k < PER; k += 4) {
      const uint4 c4 = *reinterpret_cast<const uint4*>(cnt + i0 + k);
      cv[k] = c4.x; cv[k + 1] = c4.y; cv[k + 2] = c4.z; cv[k + 3] = c4.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < PER; ++k) cv[k] = k < nrows ? cnt[i0 + k] : 0u;
  }
  if constexpr (TABLE) {  // the weights are differences of the shared prefix sums
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = i0 + k;
      wv[k] = (cv[k] != 0u) ? (uint32_t)(C[i] - (i > 0 ? C[i - 1] : 0ull)) : 1u;
    }
  }
  // even rows first, then odd rows (the gather kernel pairs lane groups of opposite row
  // parity so that their LDS reads fall in different banks); each part ascending and
  // padded to an even length with a zero row of its parity
  int ne = 0, no = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    if (cv[k] != 0u) {
      if ((i0 + k) & 1) ++no;
      else ++ne;
    }
  }
  const int cnt2 = ne | (no << 16);  // both counts <= d_in < 2^16
  const int incl2 = wave_inclusive_scan<int>(cnt2, lane);
  const int tot2 = __builtin_amdgcn_readlane(incl2, kWave - 1);
  const int NE = tot2 & 0xffff, NO = tot2 >> 16;
  const int nepad = (NE + 1) & ~1, nopad = (NO + 1) & ~1;
  int pe = (incl2 - cnt2) & 0xffff;
  int po = nepad + ((incl2 - cnt2) >> 16);
  uint2* lst = p.list + tok * list_stride(d_in);
  const int rb = gather_row_bytes(d_in);  // the gather kernel reads rows of its LDS slice
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const uint32_t c = cv[k];
    if (c) {
      const float coef = (float)(((double)c * (double)xv[k] * (double)Tw) / ((double)r * (double)wv[k]));
      const int at = ((i0 + k) & 1) ? po++ : pe++;
      lst[at] = make_uint2((uint32_t)((i0 + k) * rb), __float_as_uint(coef));
    }
  }
  if (lane == 0) {
    if (NE & 1) lst[NE] = make_uint2((uint32_t)(zero_row_even(d_in) * rb), 0u);
    if (NO & 1) lst[nepad + NO] = make_uint2((uint32_t)(zero_row_odd(d_in) * rb), 0u);
    p.ucount[tok] = (nepad << 16) | (nepad + nopad);
  }
}

template <int BF, int PER, bool TABLE>
hipError_t launch_per(const FwdParams& p, hipStream_t s) {
  const int64_t ntok = (int64_t)p.B * p.n;
  const dim3 grid((unsigned)((ntok + kWaves - 1) / kWaves));
  const size_t lds = (size_t)sample_lds_bytes(p.d_in, TABLE);
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_sample<BF, PER, TABLE>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_sample<BF, PER, TABLE>), grid, dim3(64 * kWaves), lds, s, p);
  return hipGetLastError();
}

template <int BF, int PER>
hipError_t launch_mode(const FwdParams& p, hipStream_t s) {
  return p.weight_sampling ? launch_per<BF, PER, true>(p, s) : launch_per<BF, PER, false>(p, s);
}

template <int BF>
hipError_t launch_bf(const FwdParams& p, hipStream_t s) {
  const int per = (p.d_in + kWave - 1) / kWave;
  if (per <= 4) return launch_mode<BF, 4>(p, s);
  if (per <= 8) return launch_mode<BF, 8>(p, s);
  if (per <= 12) return launch_mode<BF, 12>(p, s);
  if (per <= 16) return launch_mode<BF, 16>(p, s);
  if (per <= 24) return launch_mode<BF, 24>(p, s);
  if (per <= 32) return launch_mode<BF, 32>(p, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_sample(const FwdParams& p, hipStream_t s) {
  return p.bf16 ? launch_bf<1>(p, s) : launch_bf<0>(p, s);
}

}  // namespace mca
