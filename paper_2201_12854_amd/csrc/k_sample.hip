// Sampler of the MCA forward pass on gfx950: one wavefront per token j of batch row b.
//
//   1. column max m_j = max over the per-(head, query tile) partials written by the score
//      pass, and the sample count of Eq. 9 (Sec. "Determining Sample Size from
//      Attention") in float64: t = (len_b * m_j) / alpha, r_j = ceil(t * t) clamped to
//      [1, d_in]; padded keys get 0. r_j = d_in marks a saturated token, encoded exactly
//      by the gather kernel's MFMA path (cost of d_in samples, no error). Under local-
//      window attention the partials hold |S_q| A[q, j] (each query's key count in place
//      of n) and t = m_j / alpha.
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

constexpr int kMaxWaves = 4;  // tokens (waves) per block: 4, 2 or 1, as the LDS allows


// Orders LDS accesses of different lanes of one wavefront: the hardware executes a wave's
// LDS instructions in issue order, so only compiler reordering has to be prevented.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}



template <int BF>
__device__ __forceinline__ void write_zero4(const FwdParams& p, int64_t off) {
  if constexpr (BF) *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.Henc) + off) = make_uint2(0u, 0u);
  else *reinterpret_cast<float4*>(static_cast<float*>(p.Henc) + off) = make_float4(0.f, 0.f, 0.f, 0.f);
  if (p.enc_out) *reinterpret_cast<float4*>(p.enc_out + off) = make_float4(0.f, 0.f, 0.f, 0.f);
}

// Sum over the 64 lanes in a fixed order (DPP within rows of 16, then the four rows).
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<0xB1>(v);
  v += dpp_f32<0x4E>(v);
  v += dpp_f32<0x141>(v);
  v += dpp_f32<0x140>(v);
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (a + b) + (c + d);
}

// Median of the N = H len values v[h n + i], h < H, i < len (all non-negative floats, so
// their bit patterns order like the values): the value of rank (N - 1) / 2 (counting from
// 0), then, for even N, the mean with the next value up (the count of values <= it and the
// smallest value above it). Up to 2048 values are held in registers (32 per lane) and the
// rank is selected there; longer columns are selected by a radix select over 8-bit digits
// that reads the column again per pass.
constexpr int kSelRegs = 32;

// Value u * 64 + lane of the column (u * 64 + lane < N), read from memory.
__device__ __forceinline__ uint32_t column_at(const float* v, int n, int len, int u, int lane) {
  const int idx = u * kWave + lane, h = idx / len;
  return __float_as_uint(v[(int64_t)h * n + idx - h * len]);
}

// Radix select from memory: each pass counts the values that match the digits found so far
// in a 256-bin histogram in the wave's LDS region; the bin holding the rank gives the next
// digit, most significant first.
__device__ __forceinline__ uint32_t column_select(const float* v, int n, int len, int N, uint32_t k, uint32_t* hist,
                                                  int lane) {
  const int rounds = (N + kWave - 1) / kWave;
  uint32_t prefix = 0u, pmask = 0u;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int bb = lane; bb < 256; bb += kWave) hist[bb] = 0u;
    wave_lds_sync();
    for (int u = 0; u < rounds; ++u) {
      if (u * kWave + lane < N) {
        const uint32_t x = column_at(v, n, len, u, lane);
        if ((x & pmask) == prefix) atomicAdd(hist + ((x >> shift) & 255u), 1u);
      }
    }
    wave_lds_sync();
    const uint4 hc = *reinterpret_cast<const uint4*>(hist + 4 * lane);
    const uint32_t sum = hc.x + hc.y + hc.z + hc.w;
    const uint32_t incl = wave_inclusive_scan<uint32_t>(sum), excl = incl - sum;
    uint32_t d = 4u * lane, below = excl;  // the digit and the count below it, if k is in this lane's bins
    if (k >= below + hc.x) {
      below += hc.x;
      ++d;
      if (k >= below + hc.y) {
        below += hc.y;
        ++d;
        if (k >= below + hc.z) {
          below += hc.z;
          ++d;
        }
      }
    }
    const uint64_t own = __ballot(excl <= k && k < incl);  // exactly one lane
    const int src = __ffsll((unsigned long long)own) - 1;
    k -= (uint32_t)__shfl((int)below, src);
    prefix |= (uint32_t)__shfl((int)d, src) << shift;
    pmask |= 255u << shift;
    wave_lds_sync();  // every lane has read the histogram before the next pass clears it
  }
  return prefix;
}

// The same selection for values held in registers: the rank-k value is the largest bit
// pattern v with #{x < v} <= k, built bit by bit from the top (the sign bit of non-negative
// floats is 0); each step counts the values below the candidate with one compare and one
// wave ballot per register. Register slots past the values hold 0xffffffff, which no
// candidate exceeds. Bits hi .. lo are decided here, the ones above come in as prefix.
template <int R>
__device__ __forceinline__ uint32_t select_bits(const uint32_t (&reg)[kSelRegs], uint32_t k, uint32_t prefix, int hi,
                                                int lo) {
  for (int bit = hi; bit >= lo; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    uint32_t below = 0u;
#pragma unroll
    for (int u = 0; u < R; ++u) below += (uint32_t)__popcll(__ballot(reg[u] < cand));
    if (below <= k) prefix = cand;
  }
  return prefix;
}

// Rank-k selection of the values in the first R registers: the top 12 bits (bits 30 .. 19)
// over every value, then, when at most 256 values share those bits with the result, the
// rest over those values only, moved into at most four registers through the wave's LDS
// region buf (256 words): a value with smaller top bits is below every remaining candidate
// and a value with larger ones below none, so the rank among the shared values is k minus
// the count of smaller ones.
constexpr int kTopShift = 19;
template <int R>
__device__ __forceinline__ uint32_t column_select_regs(const uint32_t (&reg)[kSelRegs], uint32_t k, uint32_t* buf,
                                                      int lane) {
  const uint32_t prefix = select_bits<R>(reg, k, 0u, 30, kTopShift);
  const uint32_t top = prefix >> kTopShift;
  uint32_t smaller = 0u, same = 0u, mine = 0u;
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const uint32_t t = reg[u] >> kTopShift;  // padding: 0x1fff, above every top
    smaller += (uint32_t)__popcll(__ballot(t < top));
    const bool eq = t == top;
    same += (uint32_t)__popcll(__ballot(eq));
    mine += eq ? 1u : 0u;
  }
  if (same > 256u) return select_bits<R>(reg, k, prefix, kTopShift - 1, 0);
  const uint32_t incl = wave_inclusive_scan<uint32_t>(mine);
  uint32_t at = incl - mine;
#pragma unroll
  for (int u = 0; u < R; ++u)
    if ((reg[u] >> kTopShift) == top) buf[at++] = reg[u];
  wave_lds_sync();
  uint32_t r2[kSelRegs];
#pragma unroll
  for (int u = 0; u < 4; ++u) r2[u] = (uint32_t)(u * kWave + lane) < same ? buf[u * kWave + lane] : 0xffffffffu;
  wave_lds_sync();  // every lane has read buf before a later use of the region
  const uint32_t k2 = k - smaller;
  if (same <= 64u) return select_bits<1>(r2, k2, prefix, kTopShift - 1, 0);
  if (same <= 128u) return select_bits<2>(r2, k2, prefix, kTopShift - 1, 0);
  return select_bits<4>(r2, k2, prefix, kTopShift - 1, 0);
}

__device__ __forceinline__ float column_median(const float* v, int H, int n, int len, uint32_t* hist, int lane) {
  const int N = H * len;
  const bool cached = N <= kSelRegs * kWave;
  uint32_t reg[kSelRegs];
  uint32_t lo;
  if (cached) {
    // value u * 64 + lane is v[h n + i] with h = (u * 64 + lane) / len, stepped without a
    // division per value
    int h = lane / len, i = lane - h * len;
    const int dh = kWave / len, di = kWave - dh * len;  // 64 = dh len + di
#pragma unroll
    for (int u = 0; u < kSelRegs; ++u) {
      reg[u] = u * kWave + lane < N ? __float_as_uint(v[(int64_t)h * n + i]) : 0xffffffffu;
      h += dh;
      i += di;
      if (i >= len) {
        i -= len;
        ++h;
      }
    }
    const uint32_t k = (uint32_t)(N - 1) / 2;
    if (N <= 8 * kWave) lo = column_select_regs<8>(reg, k, hist, lane);
    else if (N <= 16 * kWave) lo = column_select_regs<16>(reg, k, hist, lane);
    else if (N <= 24 * kWave) lo = column_select_regs<24>(reg, k, hist, lane);
    else lo = column_select_regs<32>(reg, k, hist, lane);
  } else {
    lo = column_select(v, n, len, N, (uint32_t)(N - 1) / 2, hist, lane);
  }
  if (N % 2) return __uint_as_float(lo);
  // rank N / 2: lo again if more than N / 2 values are <= lo, else the smallest value above
  // (a register slot past N, 0xffffffff, is above every lo and counts for neither)
  uint32_t le = 0u, above = 0xffffffffu;
  if (cached) {
#pragma unroll
    for (int u = 0; u < kSelRegs; ++u) {
      le += reg[u] <= lo ? 1u : 0u;
      if (reg[u] > lo) above = min(above, reg[u]);
    }
  } else {
    const int rounds = (N + kWave - 1) / kWave;
    for (int u = 0; u < rounds; ++u) {
      if (u * kWave + lane < N) {
        const uint32_t x = column_at(v, n, len, u, lane);
        le += x <= lo ? 1u : 0u;
        if (x > lo) above = min(above, x);
      }
    }
  }
  for (int o = 32; o >= 1; o >>= 1) {  // wave sums and minima
    le += (uint32_t)__shfl_xor((int)le, o);
    above = min(above, (uint32_t)__shfl_xor((int)above, o));
  }
  const uint32_t hi = le > (uint32_t)N / 2 ? lo : above;
  return (float)(0.5 * ((double)__uint_as_float(lo) + (double)__uint_as_float(hi)));
}

// The median rule's column statistic, before the sampler: one wavefront per key j < len of
// batch row b takes the median of its H len probabilities (written key-major by the score
// pass) and leaves it in the key's first column-max partial slot, the only one the sampler
// reads under this rule. Padded keys are skipped (the sampler gives them r = 0).
constexpr int kMedWaves = 4;
__global__ __launch_bounds__(64 * kMedWaves) void k_colmedian(FwdParams p) {
  __shared__ __align__(16) uint32_t hist[kMedWaves][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t tok = (int64_t)blockIdx.x * kMedWaves + wave;
  if (tok >= (int64_t)p.B * p.n) return;  // wave-uniform; no block barrier follows
  const int b = (int)(tok / p.n), j = (int)(tok - (int64_t)b * p.n);
  int len = p.seq_lens ? p.seq_lens[b] : p.n;
  len = min(max(len, 1), p.n);
  if (j >= len) return;
  const float m = column_median(p.acol + tok * (int64_t)p.H * p.n, p.H, p.n, len, hist[wave], lane);
  if (lane == 0) p.colmax_part[tok * p.nparts] = m;
}

// Per-wave results of phase 1, shared with the block for the pooled draws.
struct TokInfo {
  int r[kMaxWaves];     // draws of the wave's token (0: no draws)
  int j[kMaxWaves], b[kMaxWaves];
  int P[kMaxWaves + 1];  // exclusive prefix sums of r: the token's first pooled draw
  uint64_t T[kMaxWaves];  // total weight C[d_in - 1]
};
constexpr int kHeader = 512;  // bytes of LDS before the per-token regions
static_assert(sizeof(TokInfo) <= kHeader, "header");

// LDS of a block: the header, then
//   Eq. 4: per wave C uint64 [d_in] (after the draws: records (x bits, w), uint32 pairs
//          [d_in]) and cnt uint32 [d_in] (after the draws: record row | count);
//   Eq. 6: the shared C uint64 [d_in], then per wave cnt uint32 [d_in] and record x
//          float32 [d_in].
__host__ __device__ inline int round16(int v) { return (v + 15) / 16 * 16; }
__host__ __device__ inline int sample_shared_bytes(int d_in, bool table) { return table ? round16(8 * d_in) : 0; }
__host__ __device__ inline int sample_region_bytes(int d_in, bool table) {
  return table ? 2 * round16(4 * d_in) : round16(8 * d_in) + round16(4 * d_in);
}
__host__ __device__ inline int sample_lds_bytes(int d_in, bool table, int nw) {
  return kHeader + sample_shared_bytes(d_in, table) + nw * sample_region_bytes(d_in, table);
}
__device__ __forceinline__ int region_off(int d_in, bool table, int w) {
  return kHeader + sample_shared_bytes(d_in, table) + w * sample_region_bytes(d_in, table);
}
__device__ __forceinline__ int c_off(int d_in, bool table, int w) { return table ? kHeader : region_off(d_in, false, w); }
__device__ __forceinline__ int cnt_off(int d_in, bool table, int w) {
  return region_off(d_in, table, w) + (table ? 0 : round16(8 * d_in));
}

// LDS reads by 32-bit LDS address (offset into the workgroup's LDS).
__device__ __forceinline__ uint32_t lds_addr_u64(const uint64_t* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint64_t*)p;  // address-space cast
}
__device__ __forceinline__ uint64_t lds_read_u64(uint32_t addr) {
  return *reinterpret_cast<__attribute__((address_space(3))) const uint64_t*>((uintptr_t)addr);
}

// W draws of one thread of the block's pool: draw d = d0 + 64 NW u (u < W) of the
// concatenated draws of the block's tokens (token w owns [P_w, P_w + r_w)). Each is draw
// k = d - P_w of its token: Philox4x32-10 with counter (k, j, b, 0), t = floor(u T / 2^64)
// and s = min{i : C_i > t}, the W searches together so that their LDS reads overlap;
// then the token's count of row s goes up by one.
template <int W, int NW, bool TABLE>
__device__ __forceinline__ void draw_batch(const FwdParams& p, const TokInfo& I, unsigned char* smem, int d0,
                                           const int* Ps, int D) {
  const int d_in = p.d_in;
  uint64_t t[W];
  int lo[W], wt[W], kk[W];
  uint32_t a[W], a0[W];  // LDS byte addresses: the search position, the token's C
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const int d = min(d0 + u * 64 * NW, D - 1);  // clamped: only d < D is counted
    int w = 0;  // the token: number of token starts P_1 .. P_{NW-1} at or below d
#pragma unroll
    for (int i = 1; i < NW; ++i) w += d >= Ps[i];
    wt[u] = w;
    kk[u] = d - I.P[w];
    const u32x4 o = philox4x32_10(u32x4{(uint32_t)kk[u], (uint32_t)I.j[w], (uint32_t)I.b[w], 0u}, p.seed_lo,
                                  p.seed_hi);
    t[u] = __umul64hi((uint64_t)o.x | ((uint64_t)o.y << 32), I.T[w]);  // in [0, T)
    a0[u] = lds_addr_u64(reinterpret_cast<const uint64_t*>(smem + c_off(d_in, TABLE, w)));
  }
  // s = #{i : C_i <= t} (C is non-decreasing and C[d_in-1] = T > t): a halving search
  // whose length sequence is the same for every lane (uniform), on LDS byte addresses
  // biased by -8 so that one add gives both the probe address and the candidate base.
  // Per step: add, 64-bit LDS read, compare, select. Step-major over the W draws so that
  // their LDS reads are in flight together.
#pragma unroll
  for (int u = 0; u < W; ++u) a[u] = a0[u] - 8;  // address of C[base - 1], base = 0
  for (int len = d_in; len > 1;) {
    const int half = len >> 1;
#pragma unroll
    for (int u = 0; u < W; ++u) {
      const uint32_t cand = a[u] + 8 * half;  // C[base + half - 1]
      a[u] = lds_read_u64(cand) <= t[u] ? cand : a[u];
    }
    len -= half;
  }
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const uint32_t at = a[u] + 8;  // C[base]
    lo[u] = (int)((at - a0[u]) >> 3) + (lds_read_u64(at) <= t[u] ? 1 : 0);
  }
#pragma unroll
  for (int u = 0; u < W; ++u) {
    if (d0 + u * 64 * NW < D) {
      const int w = wt[u];
      uint32_t* cnt = reinterpret_cast<uint32_t*>(smem + cnt_off(d_in, TABLE, w));
      atomicAdd(cnt + lo[u], 1u);
      const int64_t tok = (int64_t)I.b[w] * p.n + I.j[w];
      const int64_t o2 = tok * d_in + kk[u];
      if (p.idx_out) p.idx_out[o2] = lo[u];
      if (p.coef_out) {
        const uint64_t* Cw = reinterpret_cast<const uint64_t*>(smem + c_off(d_in, TABLE, w));
        const uint64_t ws = Cw[lo[u]] - (lo[u] > 0 ? Cw[lo[u] - 1] : 0ull);
        const double xs = p.bf16 ? (double)load_f32(static_cast<const uint16_t*>(p.X) + tok * d_in, lo[u])
                                 : (double)load_f32(static_cast<const float*>(p.X) + tok * d_in, lo[u]);
        p.coef_out[o2] = (float)((xs * (double)I.T[w]) / ((double)I.r[w] * (double)ws));
      }
    }
  }
}

// PER: upper bound of the rows one lane owns, ceil(d_in / 64) <= PER. TABLE: the
// input-independent probability of Eq. 6, whose prefix sums come from the prepared
// weights (copied into LDS once per block and shared by its tokens); otherwise the
// per-token probability of Eq. 4, quantised and scanned per token.
// Phase 1: every wave prepares its own token (count, distribution, zeroed counts).
// Phase 2: the block's draws are pooled over all its threads. Phase 3: every wave merges
// its token's counts into the list. Two block barriers separate the phases; no wave
// leaves before them.
template <int BF, int PER, bool TABLE, int NW>
__global__ __launch_bounds__(64 * NW) void k_sample(FwdParams p) {
  static_assert(NW >= 1 && NW <= kMaxWaves, "tokens per block");
  using T = typename Elem<BF>::T;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // the token's values are scalar
  const int64_t ntok = (int64_t)p.B * p.n;
  const int64_t tok = (int64_t)blockIdx.x * NW + wave;
  const int d_in = p.d_in, n = p.n;
  TokInfo& I = *reinterpret_cast<TokInfo*>(smem);
  uint64_t* C;      // this token's prefix sums (Eq. 6: the shared table)
  uint32_t* cnt;    // this token's draw counts, then record row | count
  float* rec_x;     // record x (Eq. 6)
  uint2* rec_xw;    // record (x, w) (Eq. 4)
  C = reinterpret_cast<uint64_t*>(smem + c_off(d_in, TABLE, wave));
  cnt = reinterpret_cast<uint32_t*>(smem + cnt_off(d_in, TABLE, wave));
  if constexpr (TABLE) {
    rec_x = reinterpret_cast<float*>(smem + cnt_off(d_in, true, wave) + round16(4 * d_in));
    rec_xw = nullptr;
    for (int i = threadIdx.x; i < d_in; i += 64 * NW) C[i] = p.wtable[i];
  } else {
    rec_x = nullptr;
    rec_xw = reinterpret_cast<uint2*>(C);
  }
  const bool live = tok < ntok;
  const int64_t tk = live ? tok : ntok - 1;  // a wave without a token reads a valid one
  const int b = (int)(tk / n), j = (int)(tk - (int64_t)b * n);

  // ---- phase 1. independent loads first: length, column-max partials, x (and rho under
  // Eq. 4) of this lane's contiguous run of rows [i0, i0 + nrows)
  int len = p.seq_lens ? p.seq_lens[b] : n;
  len = min(max(len, 1), n);
  const int rin = p.r_in ? p.r_in[tk] : 0;
  const float* part = p.colmax_part + tk * p.nparts;
  const bool mean_rule = p.importance == 1;
  // the token's column-max partials (column sums under the mean rule): the first eight of
  // each lane are loaded here, before x, so that all of phase 1's loads are in flight at
  // once (slots past the end re-read the last partial and count as 0)
  const bool median_rule = p.importance == 2;
  const int nparts = median_rule ? 1 : p.nparts;  // the median rule: one value, from k_colmedian
  // partial i of the token (clamped to the last): a 32-bit byte offset from the wave-uniform
  // base (nparts < 2^24), so the address needs no 64-bit arithmetic per lane
  auto part_at = [&](int i) {
    return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(part) + (uint32_t)min(i, nparts - 1) * 4u);
  };
  float pv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int t = lane + u * kWave;
    const float v = part_at(t);
    pv[u] = t < nparts ? v : 0.f;
  }
  const int per = (d_in + kWave - 1) / kWave;
  const int i0 = min(lane * per, d_in);
  const int nrows = min(per, d_in - i0);
  const T* xrow = static_cast<const T*>(p.X) + tk * d_in;
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
  // per lane in ascending order; a slot past the end adds 0 or takes the max with 0 (every
  // partial is >= 0), which leaves the result unchanged. Rows of more than 512 partials
  // continue eight at a time.
  float m = 0.f;
#pragma unroll
  for (int u = 0; u < 8; ++u) m = mean_rule ? m + pv[u] : fmaxf(m, pv[u]);
  for (int t0 = lane + 8 * kWave; t0 < nparts; t0 += 8 * kWave) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0 + u * kWave;
      const float v = part_at(t);
      pv[u] = t < nparts ? v : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) m = mean_rule ? m + pv[u] : fmaxf(m, pv[u]);
  }
  if (mean_rule) {  // the partials are column sums: the mean over H len values
    m = (float)((double)wave_sum(m) / ((double)p.H * (double)len));
  } else if (median_rule) {  // the key's median, as k_colmedian left it (a NaN stays NaN)
    m = __shfl(pv[0], 0);
  } else {
    m = wave_max(m);
  }
  if constexpr (TABLE) __syncthreads();  // the shared table is in LDS

  // 1a. sample count (Eq. 9)
  int r;
  if (j >= len) {
    r = 0;
    m = 0.f;
  } else if (p.r_in) {
    r = min(max(rin, 0), d_in);
  } else {
    // full attention: t = (len m) / alpha (Eq. 9); local window: m already carries each
    // query's key count |S_q| (the per-row n of Eq. 9), so t = m / alpha
    const double t = (p.band_half > 0 ? (double)m : (double)len * (double)m) / p.alpha;
    const double tt = t * t;
    // a t^2 that is not below d_in (a NaN too: non-finite scores) saturates the token
    r = !(tt < (double)d_in) ? d_in : max((int)ceil(tt), 1);
  }
  if (live && lane == 0) {
    p.r[tok] = r;
    if (p.colmax_out) p.colmax_out[tok] = m;
  }
  // 1b. the distribution: per-token fixed-point weights and their prefix sums (Eq. 4), or
  // the shared table (Eq. 6). No distribution (x_j = 0 under Eq. 4, W_v = 0 under Eq. 6,
  // non-finite weights) or a padded key: H~[j] = 0. A saturated token (r = d_in) is
  // encoded exactly by the gather kernel's MFMA path and has no list either.
  uint32_t wv[PER];
  uint64_t Tw = 0;
  bool none;
  if constexpr (TABLE) {
    Tw = C[d_in - 1];
    none = Tw == 0;
  } else {
    const float vmax = wave_max(lmax);
    none = !(vmax > 0.f) || !(vmax <= 3.40282347e38f);
    if (!none && r > 0 && !exact_token(r, d_in, p.exact_from)) {
      int e;
      (void)frexpf(vmax, &e);  // vmax = f 2^e, f in [0.5, 1)
      const int shift = 32 - e;
      uint64_t lsum = 0;
      if (full) {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          wv[k] = (uint32_t)ldexpf(vv[k], shift);
          lsum += wv[k];
        }
      } else {
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          wv[k] = (k < nrows) ? (uint32_t)ldexpf(vv[k], shift) : 0u;
          lsum += wv[k];
        }
      }
      const uint64_t incl = wave_inclusive_scan<uint64_t>(lsum);
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
  const bool exact = exact_token(r, d_in, p.exact_from);  // encoded on MFMA by the gather or its own kernel
  const bool sampled = live && r > 0 && !exact && !none;
  if (live && !sampled) {
    if (lane == 0) p.ucount[tok] = 0;
    if (!exact)
      for (int c = 4 * lane; c < p.d_out; c += 4 * kWave) write_zero4<BF>(p, tok * p.d_out + c);
  }
  if (sampled) {
    if (full) {
#pragma unroll
      for (int k = 0; k < PER; k += 4) *reinterpret_cast<uint4*>(cnt + i0 + k) = make_uint4(0u, 0u, 0u, 0u);
    } else {
#pragma unroll
      for (int k = 0; k < PER; ++k)
        if (k < nrows) cnt[i0 + k] = 0u;
    }
  }
  if (lane == 0) {
    I.r[wave] = sampled ? r : 0;
    I.j[wave] = j;
    I.b[wave] = b;
    I.T[wave] = Tw;
  }
  __syncthreads();

  if (threadIdx.x == 0) {  // where each token's draws start in the pool
    int acc = 0;
    for (int w = 0; w < NW; ++w) {
      I.P[w] = acc;
      acc += I.r[w];
    }
    I.P[NW] = acc;
  }
  __syncthreads();

  // ---- phase 2. the block's draws, 64 NW threads, up to 4 per thread in flight
  {
    int Ps[NW];  // block-uniform: scalar registers
#pragma unroll
    for (int i = 0; i < NW; ++i) Ps[i] = __builtin_amdgcn_readfirstlane(I.P[i]);
    const int D = __builtin_amdgcn_readfirstlane(I.P[NW]);
    const int nper = (D + 64 * NW - 1) / (64 * NW);
    for (int u0 = 0; u0 < nper; u0 += 4) {
      const int d0 = threadIdx.x + u0 * 64 * NW;
      const int w = min(4, nper - u0);
      if (w == 4) draw_batch<4, NW, TABLE>(p, I, smem, d0, Ps, D);
      else if (w == 3) draw_batch<3, NW, TABLE>(p, I, smem, d0, Ps, D);
      else if (w == 2) draw_batch<2, NW, TABLE>(p, I, smem, d0, Ps, D);
      else draw_batch<1, NW, TABLE>(p, I, smem, d0, Ps, D);
    }
  }
  __syncthreads();
  if (!sampled) return;

  // ---- phase 3. merge duplicates into the token's list: even rows first, then odd rows
  // (the gather kernel pairs lane groups of opposite row parity so that their LDS reads
  // fall in different banks), each part ascending and padded to an even length with a zero
  // row of its parity. The owners of the rows write compact records (row | count, x, w) in
  // list order; then each lane turns records lane, lane + 64, ... into list entries.
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
  // full rows with PER even: every lane's run starts on an even row, so row i0 + k has the
  // parity of k (known at compile time)
  const bool even_runs = full && PER % 2 == 0;
  const auto odd_static = [](int k) { return (k & 1) != 0; };
  const auto odd_lane = [&](int k) { return ((i0 + k) & 1) != 0; };
  int ne = 0, no = 0;
  auto count = [&](auto odd) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (cv[k] != 0u) {
        if (odd(k)) ++no;
        else ++ne;
      }
    }
  };
  if (even_runs) count(odd_static);
  else count(odd_lane);
  const int cnt2 = ne | (no << 16);  // both counts <= d_in < 2^16
  const int incl2 = (int)wave_inclusive_scan<uint32_t>((uint32_t)cnt2);
  const int tot2 = __builtin_amdgcn_readlane(incl2, kWave - 1);
  const int NE = tot2 & 0xffff, NO = tot2 >> 16, U = NE + NO;
  int pe = (incl2 - cnt2) & 0xffff;
  int po = NE + ((incl2 - cnt2) >> 16);
  wave_lds_sync();  // every lane has its counts before the records overwrite them
  auto records = [&](auto odd) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const uint32_t c = cv[k];
      if (c) {
        const int at = odd(k) ? po++ : pe++;
        cnt[at] = (uint32_t)(i0 + k) | (c << 16);
        if constexpr (TABLE) rec_x[at] = xv[k];
        else rec_xw[at] = make_uint2(__float_as_uint(xv[k]), wv[k]);
      }
    }
  };
  if (even_runs) records(odd_static);
  else records(odd_lane);
  wave_lds_sync();
  const int nepad = (NE + 1) & ~1, nopad = (NO + 1) & ~1;
  uint2* lst = p.list + tok * list_stride(d_in);
  const int rb = gather_row_bytes(d_in);  // the gather kernel reads rows of its LDS slice
  for (int q = lane; q < U; q += kWave) {
    const uint32_t e = cnt[q];
    const int row = (int)(e & 0xffffu);
    const uint32_t c = e >> 16;
    float x;
    uint32_t w;
    if constexpr (TABLE) {
      x = rec_x[q];
      w = (uint32_t)(C[row] - (row > 0 ? C[row - 1] : 0ull));
    } else {
      const uint2 xw = rec_xw[q];
      x = __uint_as_float(xw.x);
      w = xw.y;
    }
    const float coef = (float)(((double)c * (double)x * (double)Tw) / ((double)r * (double)w));
    lst[q < NE ? q : q + (nepad - NE)] = make_uint2((uint32_t)(row * rb), __float_as_uint(coef));
  }
  if (lane == 0) {
    if (NE & 1) lst[NE] = make_uint2((uint32_t)(zero_row_even(d_in) * rb), 0u);
    if (NO & 1) lst[nepad + NO] = make_uint2((uint32_t)(zero_row_odd(d_in) * rb), 0u);
    p.ucount[tok] = (nepad << 16) | (nepad + nopad);
  }
}

template <int BF, int PER, bool TABLE, int NW>
hipError_t launch_nw(const FwdParams& p, hipStream_t s) {
  const int64_t ntok = (int64_t)p.B * p.n;
  const dim3 grid((unsigned)((ntok + NW - 1) / NW));
  const size_t lds = (size_t)sample_lds_bytes(p.d_in, TABLE, NW);
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_sample<BF, PER, TABLE, NW>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  return launch_stage_kernel(k_sample<BF, PER, TABLE, NW>, grid, dim3(64 * NW), lds, s, p);
}

// As many tokens per block as the LDS holds (16, 8 or 4): more tokens per block spread the
// pooled draws over more threads.
template <int BF, int PER, bool TABLE>
hipError_t launch_per(const FwdParams& p, hipStream_t s) {
  constexpr int kLds = 160 * 1024;
  // four tokens per block: several blocks per CU, so that one block's first loads overlap
  // another's draws (measured faster than 16 or 8 tokens per block, which balance the
  // pooled draws over more tokens, at the BERT-base, BERT-large, long-sequence and
  // local-window shapes)
  if (sample_lds_bytes(p.d_in, TABLE, 4) <= kLds) return launch_nw<BF, PER, TABLE, 4>(p, s);
  if (sample_lds_bytes(p.d_in, TABLE, 2) <= kLds) return launch_nw<BF, PER, TABLE, 2>(p, s);
  if (sample_lds_bytes(p.d_in, TABLE, 1) <= kLds) return launch_nw<BF, PER, TABLE, 1>(p, s);
  return hipErrorInvalidValue;
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
  if (p.importance != 2) return p.bf16 ? launch_bf<1>(p, s) : launch_bf<0>(p, s);
  // the median rule: k_colmedian, then the sampler; a profiler's event pair spans both
  FwdParams p1 = p, p2 = p;
  p1.ev_stop = nullptr;
  p2.ev_start = nullptr;
  const int64_t ntok = (int64_t)p.B * p.n;
  const dim3 grid((unsigned)((ntok + kMedWaves - 1) / kMedWaves));
  const hipError_t e = launch_stage_kernel(k_colmedian, grid, dim3(64 * kMedWaves), 0, s, p1);
  if (e != hipSuccess) return e;
  return p.bf16 ? launch_bf<1>(p2, s) : launch_bf<0>(p2, s);
}

}  // namespace mca
