// Exact encoding of saturated tokens (r_j = d_in): H~[j] = x_j W_v on MFMA.
//
// The count rule of Eq. 9 can ask for more samples than W_v has rows; such a token is
// encoded exactly, which costs what d_in samples would and has no error, so the error
// bounds of Lemma 1 / Theorem 1 still hold.
//
// A block scans 256 consecutive tokens, compacts the saturated ones and computes their
// H~ rows for 64 columns with 16x16 MFMA tiles. Operand tiles go through LDS so each
// global load is shared by the four waves; both operands are k-contiguous rows: x, and
// the prepared transposed W_v^T (zero padded to a multiple of 32 along k).
#include <type_traits>

#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kRange = 256;  // tokens scanned per block
constexpr int kRows = 64;    // saturated tokens per tile (4 waves x 16)
constexpr int kCols = 64;    // output columns per block (4 MFMA column tiles)
constexpr int kPad = 8;      // LDS row padding (16-bit elements)
constexpr int kDepth = 4;    // k-steps of operand tiles in flight in registers

template <int BF>
__device__ __forceinline__ void store_out(const FwdParams& p, int64_t off, float v) {
  if constexpr (BF) static_cast<uint16_t*>(p.Henc)[off] = (uint16_t)f32_to_bf16_bits(v);
  else static_cast<float*>(p.Henc)[off] = v;
  if (p.enc_out) p.enc_out[off] = v;
}

// Compacts the saturated tokens of [t0, t0 + 256) into sl[] in ascending order and
// returns their number. Contains barriers.
__device__ __forceinline__ int compact_saturated(const FwdParams& p, int64_t t0, int* sl, int* wcnt, int tid) {
  const int lane = tid & 63, wave = tid >> 6;
  const int64_t tok = t0 + tid;
  const bool sat = tok < (int64_t)p.B * p.n && p.r[tok] >= p.d_in;
  const uint64_t mask = __ballot(sat);
  if (lane == 0) wcnt[wave] = __popcll(mask);
  lds_barrier();
  int base = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) base += wcnt[w];
    total += wcnt[w];
  }
  if (sat) sl[base + __popcll(mask & ((1ull << lane) - 1ull))] = tid;
  lds_barrier();
  return total;
}

// One k-step of 16-byte chunks: bf16 = 8 k, fp32 = 4 k. A k-step spans 4 chunks (32 bf16 or
// 16 fp32 k); thread (row = tid / 4, chunk = tid % 4) stages one chunk of the x tile and
// one of the W_v^T tile per step. Rows past d_in read zeros (x guarded, W_v^T padded).
template <int BF>
__device__ __forceinline__ uint4 load_x_chunk(const void* xrow_v, int k, int d_in, bool xvec) {
  if constexpr (BF) {
    const uint16_t* x = static_cast<const uint16_t*>(xrow_v);
    if (xvec && k + 8 <= d_in) return *reinterpret_cast<const uint4*>(x + k);
    uint32_t e16[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) e16[e] = (k + e < d_in) ? x[k + e] : 0u;
    return make_uint4(e16[0] | (e16[1] << 16), e16[2] | (e16[3] << 16), e16[4] | (e16[5] << 16), e16[6] | (e16[7] << 16));
  } else {
    const float* x = static_cast<const float*>(xrow_v);
    if (xvec && k + 4 <= d_in) return *reinterpret_cast<const uint4*>(x + k);
    uint32_t h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = (k + e < d_in) ? __float_as_uint(x[k + e]) : 0u;
    return make_uint4(h[0], h[1], h[2], h[3]);
  }
}

// Grid: (ranges of 256 consecutive tokens) x (64-column blocks of d_out). A block reads
// the sample counts of its tokens, compacts the saturated ones (no device-side list and
// no counters), then for every group of 64 of them computes the 64 x 64 output tile:
// x and W_v^T tiles of one k-step are staged in LDS (double buffered, one barrier per
// step, coalesced 16-byte loads issued four steps ahead), and wave w multiplies rows 16 w .. 16 w + 15 against
// the 4 column tiles with
//   bf16: v_mfma_f32_16x16x32_bf16 (lane group g: k = 8 g .. 8 g + 7 of the step)
//   fp32: v_mfma_f32_16x16x4f32    (lane group g: k = 4 g .. 4 g + 3, one MFMA per k)
template <int BF, bool FAST>
__global__ __launch_bounds__(kThreads) void k_dense_encode(FwdParams p) {
  constexpr int KS = BF ? 32 : 16;               // k per step
  constexpr int RW = BF ? 32 + kPad : 32 + kPad;  // LDS row length in 16-bit units (64 bytes + pad)
  __shared__ int sl[kRange];
  __shared__ int wcnt[kWaves];
  __shared__ __align__(16) uint16_t As[2][kRows][RW];
  __shared__ __align__(16) uint16_t Bs[2][kCols][RW];
  const int64_t t0 = (int64_t)blockIdx.x * kRange;
  const int c0 = blockIdx.y * kCols;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int nsat = compact_saturated(p, t0, sl, wcnt, tid);
  if (nsat == 0) return;
  const int d_in = p.d_in, d_out = p.d_out;
  const int64_t dpad = p.din_pad;
  const bool xvec = (d_in & (BF ? 7 : 3)) == 0;
  const int nks = (d_in + KS - 1) / KS;
  const int lr = tid >> 2, lc = tid & 3;  // staging: tile row, 16-byte chunk
  const char* X = static_cast<const char*>(p.X);
  const int esz = BF ? 2 : 4;
  const char* wrow = static_cast<const char*>(p.Wt) + ((int64_t)(c0 + lr) * dpad) * esz + lc * 16;

  for (int m0 = 0; m0 < nsat; m0 += kRows) {
    // rows past the last saturated token repeat a valid row; their outputs are not stored
    const int slot = m0 + lr;
    const char* xrow = X + (t0 + sl[slot < nsat ? slot : 0]) * (int64_t)d_in * esz;
    f32x4_t acc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // register ring: the tiles of the next kDepth k-steps are in flight while one is used.
    // FAST (d_in a multiple of kDepth k-steps): plain vector loads, the prefetch index
    // clamped to the last step, so the loop body has no branches at all.
    auto load_a = [&](int ks) -> uint4 {
      if constexpr (FAST) return *reinterpret_cast<const uint4*>(xrow + (int64_t)ks * 64 + lc * 16);
      else return load_x_chunk<BF>(xrow, ks * KS + lc * (16 / esz), d_in, xvec);
    };
    auto load_b = [&](int ks) -> uint4 { return *reinterpret_cast<const uint4*>(wrow + (int64_t)ks * 64); };
    uint4 ra[kDepth], rb[kDepth];
#pragma unroll
    for (int t = 0; t < kDepth; ++t) {
      const int kk = t < nks ? t : nks - 1;
      ra[t] = load_a(kk);
      rb[t] = load_b(kk);
    }
    for (int ks0 = 0; ks0 < nks; ks0 += kDepth) {
#pragma unroll
      for (int t = 0; t < kDepth; ++t) {
        const int ks = ks0 + t;
        // FAST: nks is a multiple of kDepth, so every step of the ring exists (no branch)
        if (FAST || ks < nks) {
          const int buf = t & 1;
          *reinterpret_cast<uint4*>(&As[buf][lr][lc * 8]) = ra[t];
          *reinterpret_cast<uint4*>(&Bs[buf][lr][lc * 8]) = rb[t];
          lds_barrier();
          const int kn = ks + kDepth < nks ? ks + kDepth : nks - 1;
          ra[t] = load_a(kn);
          rb[t] = load_b(kn);
          const uint4 a = *reinterpret_cast<const uint4*>(&As[buf][wave * 16 + r16][8 * g]);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const uint4 b = *reinterpret_cast<const uint4*>(&Bs[buf][16 * c + r16][8 * g]);
            if constexpr (BF) {
              acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                              __builtin_bit_cast(bf16x8_t, b), acc[c], 0, 0, 0);
            } else {
              acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc[c], 0, 0, 0);
              acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc[c], 0, 0, 0);
              acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc[c], 0, 0, 0);
              acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc[c], 0, 0, 0);
            }
          }
        }
      }
    }
    // acc[c][i] = H~[saturated token m0 + 16 w + 4 g + i][column c0 + 16 c + l % 16]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int s2 = m0 + wave * 16 + 4 * g + i;
      if (s2 < nsat) {
        const int64_t base = (t0 + sl[s2]) * d_out + c0 + r16;
#pragma unroll
        for (int c = 0; c < 4; ++c) store_out<BF>(p, base + 16 * c, acc[c][i]);
      }
    }
    lds_barrier();  // the next group reuses the LDS buffers
  }
}

}  // namespace

hipError_t launch_dense_encode(const FwdParams& p, hipStream_t s) {
  const int64_t tokens = (int64_t)p.B * p.n;
  if (p.d_out % kCols != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((tokens + kRange - 1) / kRange), p.d_out / kCols);
  // fast path: whole k-steps (no ragged tail) and a whole number of prefetch rounds
  const bool fast = p.bf16 ? (p.d_in % (32 * kDepth) == 0) : (p.d_in % (16 * kDepth) == 0);
  if (p.bf16) {
    if (fast) hipLaunchKernelGGL((k_dense_encode<1, true>), grid, dim3(kThreads), 0, s, p);
    else hipLaunchKernelGGL((k_dense_encode<1, false>), grid, dim3(kThreads), 0, s, p);
  } else {
    if (fast) hipLaunchKernelGGL((k_dense_encode<0, true>), grid, dim3(kThreads), 0, s, p);
    else hipLaunchKernelGGL((k_dense_encode<0, false>), grid, dim3(kThreads), 0, s, p);
  }
  return hipGetLastError();
}

}  // namespace mca
