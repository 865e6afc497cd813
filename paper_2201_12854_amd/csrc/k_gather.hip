// Value encoding of the MCA forward pass on gfx950: H~[j] for every token that is not
// padded or zero, one column slice of W_v per block.
//
//   sampled token (0 < r_j < d_in): H~[j] = sum over its distinct sampled rows i of
//     coef_i W_v[i, :] (Eq. 2 with duplicates merged; Eq. 5 inner sum), float32
//     accumulation;
//   saturated token (r_j = d_in): H~[j] = x_j W_v exactly, on MFMA (16 tokens per tile),
//     here when the slice's B operand fits in LDS next to it (bfloat16, d_in <= 768),
//     otherwise in the kernels of the saturated-token section below (their own launch).
//
// The slice W_v[:, c0 .. c0 + WC) is converted to float32 once and kept in LDS for the
// whole block (768 x 32 floats = 96 KB: the 160 KB LDS of a gfx950 CU holds it), so the
// gather reads LDS instead of L2. A row of the slice is LPR = WC / 4 chunks of 16 bytes; a
// wave works on 64 / LPR sampled tokens at once, one per group of LPR lanes. Every lane
// takes its own pair of list entries (LDS byte offset of the row, coefficient) per round,
// loaded two rounds ahead with one coalesced 16-byte load, reads both rows whole and
// accumulates all WC columns. Each list holds its even rows first and its odd rows second
// (even and odd rows lie in opposite halves of the LDS banks); half of a group's lanes take
// the even part, half the odd part, and the chunk each lane reads at a step is permuted by
// lane and group so that the 16 lanes the LDS serves together never share a bank. A
// reduce-scatter within the group (DPP) ends the item.
//
// Work distribution: the blocks of a slice split the tokens into contiguous ranges. A block
// reads r and the list layout of its range, puts the saturated tokens on one LDS list and
// sorts the sampled tokens by the longer part of their list (key floor(8 log2), longest
// first) with LDS atomics; its waves then take work items from an LDS counter: groups of
// 16 saturated tokens first (the heaviest items), then groups of sampled tokens of
// similar length, longest first, so that the lanes of a wave and the waves of a block
// finish close together. No global atomics; outputs do not depend on which wave computes
// them.
#include <atomic>

#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };

constexpr int kThreads = 1024;


template <int BF>
__device__ __forceinline__ void store_h(const FwdParams& p, int64_t off, float v) {
  if constexpr (BF) static_cast<uint16_t*>(p.Henc)[off] = (uint16_t)f32_to_bf16_bits(v);
  else static_cast<float*>(p.Henc)[off] = v;
  if (p.enc_out) p.enc_out[off] = v;
}

template <int BF>
__device__ __forceinline__ void store_h4(const FwdParams& p, int64_t off, float4 v) {
  if constexpr (BF) {
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.Henc) + off) =
        make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(p.Henc) + off) = v;
  }
  if (p.enc_out) *reinterpret_cast<float4*>(p.enc_out + off) = v;
}

// 16 bytes of row `x` starting at element k: 8 bf16 or 4 float32; elements at or past d_in
// read as zero. VEC: d_in is a multiple of the chunk, so a chunk is all in or all out.
// Addresses are clamped into the row and the zeros selected afterwards (no branches).
template <int BF, bool VEC>
__device__ __forceinline__ uint4 load_x_chunk(const void* xrow_v, int k, int d_in) {
  constexpr int E = BF ? 8 : 4;
  if constexpr (VEC) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const char*>(xrow_v) + (int64_t)min(k, d_in - E) * (BF ? 2 : 4));
    const uint32_t keep = k < d_in ? 0xffffffffu : 0u;  // a mask keeps the load unconditional
    return make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep);
  } else {
    uint32_t h[E];
    if constexpr (BF) {
      const uint16_t* x = static_cast<const uint16_t*>(xrow_v);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t v = x[min(k + e, d_in - 1)];
        h[e] = v & ((k + e < d_in) ? 0xffffu : 0u);
      }
      return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    } else {
      const float* x = static_cast<const float*>(xrow_v);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const uint32_t v = __float_as_uint(x[min(k + e, d_in - 1)]);
        h[e] = v & ((k + e < d_in) ? 0xffffffffu : 0u);
      }
      return make_uint4(h[0], h[1], h[2], h[3]);
    }
  }
}

// Exact encoding of saturated tokens 16 gi .. 16 gi + 15 of the list for the slice's
// columns: D = X_tile W_v[:, slice] with A = x rows (k-contiguous) and B = the prepared
// W_v^T in fragment order (one coalesced 1 KB load per tile and step), both read from
// global memory.
//   bf16: v_mfma_f32_16x16x32_bf16, lane group g holds k = 32 ks + 8 g .. + 7
//   fp32: v_mfma_f32_16x16x4f32, a 16-byte chunk k = 16 ks + 4 g .. + 3 feeds 4 MFMAs
template <int BF, int WC, bool VEC>
__device__ void saturated_group(const FwdParams& p, const int* satl, int64_t t0, int gi, int nsat, int c0, int lane) {
  using T = typename Elem<BF>::T;
  constexpr int NC = WC / 16;     // 16-column MFMA tiles
  constexpr int KS = BF ? 32 : 16;  // k per step
  const int r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in;
  const int din_pad = p.din_pad;
  // rows past the list repeat a token (their results are not stored)
  const int64_t tk = t0 + satl[min(16 * gi + r16, nsat - 1)];
  const T* xrow = static_cast<const T*>(p.X) + (int64_t)tk * d_in;
  // B operand: W_v^T in fragment order, lane's 16 bytes of (tile c0 / 16 + c, step ks) at
  // ((tile * nks + ks) * 64 + lane) * E elements
  constexpr int E = BF ? 8 : 4;
  const T* wt = static_cast<const T*>(p.Wt) + ((int64_t)(c0 / 16) * (din_pad / KS) * 64 + lane) * E;
  const int nks = din_pad / KS;
  f32x4_t acc[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // rounds of RD steps, software pipelined (16-byte x loads): the loads of round t + 1 are
  // issued before the MFMAs of round t. din_pad is a multiple of 128 elements, so every round is whole and
  // the loop has no conditional code (the padded k carry zero weights; x past d_in reads
  // as zero); the round after the last reloads the last one (unused).
  constexpr int RD = VEC ? 2 : 4;
  const int nrounds = nks / RD;
  uint4 a0[RD], w0[RD][NC], a1[RD], w1[RD][NC];
#define MCA_LOAD_ROUND(A, Wr, RND)                                                              \
  _Pragma("unroll") for (int u = 0; u < RD; ++u) {                                             \
    const int ks = (RND) * RD + u;                                                             \
    A[u] = load_x_chunk<BF, VEC>(xrow, ks * KS + (BF ? 8 : 4) * g, d_in);                      \
    _Pragma("unroll") for (int c = 0; c < NC; ++c)                                             \
      Wr[u][c] = *reinterpret_cast<const uint4*>(wt + ((int64_t)c * nks + ks) * 64 * E);       \
  }
#define MCA_MFMA_ROUND(A, Wr)                                                                   \
  _Pragma("unroll") for (int u = 0; u < RD; ++u) {                                             \
    _Pragma("unroll") for (int c = 0; c < NC; ++c) {                                           \
      if constexpr (BF) {                                                                      \
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A[u]),   \
                                                        __builtin_bit_cast(bf16x8_t, Wr[u][c]), \
                                                        acc[c], 0, 0, 0);                       \
      } else {                                                                                 \
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u].x), __uint_as_float(Wr[u][c].x), acc[c], 0, 0, 0); \
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u].y), __uint_as_float(Wr[u][c].y), acc[c], 0, 0, 0); \
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u].z), __uint_as_float(Wr[u][c].z), acc[c], 0, 0, 0); \
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u].w), __uint_as_float(Wr[u][c].w), acc[c], 0, 0, 0); \
      }                                                                                        \
    }                                                                                          \
  }
  if constexpr (VEC) {
    MCA_LOAD_ROUND(a0, w0, 0)
    for (int rd = 0; rd < nrounds; rd += 2) {  // nrounds is even (nks is a multiple of 4)
      MCA_LOAD_ROUND(a1, w1, rd + 1)
      __builtin_amdgcn_sched_barrier(0);  // the next round's loads stay ahead of these MFMAs
      MCA_MFMA_ROUND(a0, w0)
      MCA_LOAD_ROUND(a0, w0, min(rd + 2, nrounds - 1))
      __builtin_amdgcn_sched_barrier(0);
      MCA_MFMA_ROUND(a1, w1)
    }
  } else {  // element-wise x loads take more registers: one buffer
    for (int rd = 0; rd < nrounds; ++rd) {
      MCA_LOAD_ROUND(a0, w0, rd)
      MCA_MFMA_ROUND(a0, w0)
    }
  }
#undef MCA_LOAD_ROUND
#undef MCA_MFMA_ROUND
  // acc[c][i] = H~[token of list row 4 g + i][c0 + 16 c + r16]; lane 4 g + i holds that token
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t tok_i = t0 + satl[min(16 * gi + 4 * g + i, nsat - 1)];
    if (16 * gi + 4 * g + i < nsat) {
      const int64_t base = (int64_t)tok_i * p.d_out + c0 + r16;
#pragma unroll
      for (int c = 0; c < NC; ++c) store_h<BF>(p, base + 16 * c, acc[c][i]);
    }
  }
}

// The same for bfloat16 with d_in <= 768 and 16-byte x loads, with the B operand (the
// slice's two 16-column tiles of the prepared W_v^T, fragment order) copied into LDS once
// per block: the x chunks of (at most 24) k steps are loaded in two batches of 12, so an
// item waits for global memory twice; steps past din_pad / 32 read zero x (k >= d_in) and
// the last B fragment.
constexpr int kLdsbSteps = 24;  // din_pad <= 768
__device__ void saturated_group_ldsb(const FwdParams& p, const int* satl, int64_t t0, int gi, int nsat, int c0,
                                     int lane, const uint4* Bl) {
  const int r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in;
  const int nks = p.din_pad / 32;
  const int64_t tk = t0 + satl[min(16 * gi + r16, nsat - 1)];
  const uint16_t* xrow = static_cast<const uint16_t*>(p.X) + (int64_t)tk * d_in;
  constexpr int HALF = kLdsbSteps / 2;
  // the chunk offsets depend only on the lane: kept inside the item (an empty asm hides the
  // value), or the compiler keeps all 24 addresses alive across the item loop
  int kb = 8 * g;
  asm volatile("" : "+v"(kb));
  const uint16_t* xr = xrow + kb;
  const int klast = d_in - 8 - kb;  // last in-row chunk start, relative to kb
  f32x4_t acc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int h0 = 0; h0 < kLdsbSteps; h0 += HALF) {
    uint4 a[HALF];
#pragma unroll
    for (int u = 0; u < HALF; ++u) {
      const int k = (h0 + u) * 32;  // relative to kb; past the row reads zero
      const uint4 v = *reinterpret_cast<const uint4*>(xr + min(k, klast));
      const uint32_t keep = k <= klast ? 0xffffffffu : 0u;
      a[u] = make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep);
    }
#pragma unroll
    for (int u = 0; u < HALF; ++u) {
      const int ks = min(h0 + u, nks - 1);
#pragma unroll
      for (int c = 0; c < 2; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[u]),
                                                        __builtin_bit_cast(bf16x8_t, Bl[(c * nks + ks) * 64 + lane]),
                                                        acc[c], 0, 0, 0);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t tok_i = t0 + satl[min(16 * gi + 4 * g + i, nsat - 1)];
    if (16 * gi + 4 * g + i < nsat) {
      const int64_t base = (int64_t)tok_i * p.d_out + c0 + r16;
#pragma unroll
      for (int c = 0; c < 2; ++c) store_h<1>(p, base + 16 * c, acc[c][i]);
    }
  }
}

// Max / min over the 64 lanes, returned in a scalar register.
__device__ __forceinline__ int wave_max_int(int v) {
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true));
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

constexpr int kChunk = kThreads;  // tokens classified per block pass (one per thread)
constexpr int kNumKeys = 96;      // sort keys floor(8 log2 M) for 1 <= M < 4096

// floor(8 log2 M) for 1 <= M < 4096 (M: the longer part of a token's list, which sets the
// rounds its lane group runs): the octave and the next three bits.
__device__ __forceinline__ int sort_key(int M) {
  const int e = 31 - __clz(M);
  const int f = e >= 3 ? (M >> (e - 3)) & 7 : (M << (3 - e)) & 7;
  return 8 * e + f;
}

// counters: [0] saturated, [1] work queue, [2 + key] key counts, [kCtrOff + key] key
// offsets, [kCtrOff + kNumKeys] sampled
constexpr int kCtrOff = 128;
constexpr int kNumCtr = 256;

__host__ __device__ inline size_t gather_lds_bytes(int d_in, int wc, bool ldsb) {
  return 128                                 // alignment of the slice
         + (size_t)(d_in + 2) * wc * 4       // W_v slice, float32, and two zero rows
         + (ldsb ? (size_t)2 * kLdsbSteps * 1024 : 0)  // B fragments of the MFMA path
         + (size_t)kChunk * 4 * 2            // sampled order, saturated list
         + kNumCtr * 4;                      // counters
}

// LDS reads by 32-bit LDS address (offset into the workgroup's LDS).
typedef __attribute__((address_space(3))) const float4 lds_float4;
__device__ __forceinline__ float4 lds_read4(uint32_t addr) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass never runs device code
  return *reinterpret_cast<lds_float4*>((uintptr_t)addr);
#else
  return float4{};
#endif
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const unsigned char*)p;  // address-space cast
}

// Entry pairs are read through a pointer that advances one round (LPR entries) at a time,
// up to three rounds past the end of a part: those entries are masked, and the list buffer
// has slack after the last token's slot so that the reads stay inside it.
__device__ __forceinline__ uint4 entry_mask(uint4 v, bool in_part, uint32_t zero_row) {
  const uint32_t k = in_part ? 0xffffffffu : 0u;
  return make_uint4((v.x & k) | (zero_row & ~k), v.y & k, (v.z & k) | (zero_row & ~k), v.w & k);
}

// acc[c] += coef * chunk (c ^ v) of a slice row: a_cl = LDS address of the row + 16 v
// (rows are RB-aligned, so bits 4.. of a_cl hold v). LPR 16-byte reads, then the FMAs.
template <int LPR>
__device__ __forceinline__ void row_fma(float4* acc, uint32_t a_cl, float coef) {
  float4 w[LPR];
#pragma unroll
  for (int c = 0; c < LPR; ++c) w[c] = lds_read4(a_cl ^ (uint32_t)(c << 4));
#pragma unroll
  for (int c = 0; c < LPR; ++c) {
    acc[c].x = fmaf(coef, w[c].x, acc[c].x);
    acc[c].y = fmaf(coef, w[c].y, acc[c].y);
    acc[c].z = fmaf(coef, w[c].z, acc[c].z);
    acc[c].w = fmaf(coef, w[c].w, acc[c].w);
  }
}

// Order entry of a sampled token: (local token << 22) | (list length << 10) | (even part / 2).
constexpr int kTokShift = 22, kLenShift = 10;

// G = 64 / LPR sampled tokens s0 .. s0 + G - 1 of the sorted order, one per group of LPR
// lanes. Lanes cl < LPR / 2 of a group take the even part of its token's list, the others
// the odd part; round t gives lane cl the entries 2 h + LPR t, + 1 of its part (h = cl mod
// LPR / 2). The lane reads chunk c ^ v of both rows at step c (v = cl, or cl ^ LPR / 2 in
// odd groups) and adds coef * chunk into acc[c]. The two groups the LDS serves together
// then read 2 LPR distinct (row parity, chunk) pairs, i.e. distinct banks. A reduce-scatter
// butterfly over the group (partners v ^ 4, v ^ 2, v ^ 1) leaves chunk v in lane cl: the
// same addition tree over the lanes' partial sums wherever the token sits, so a token's
// H~ does not depend on the other tokens of its item.
template <int BF, int RB>
__device__ void sampled_item(const FwdParams& p, const float* Ws, const uint32_t* order, int s0, int nsampled,
                             int64_t t0, int c0, int lane) {
  constexpr int LPR = RB / 16;  // lanes per group, 16-byte chunks per slice row
  constexpr int HALF = LPR / 2;
  static_assert(LPR == 4 || LPR == 8, "slice rows of 64 or 128 bytes");
  const int g = lane / LPR, cl = lane % LPR;
  const bool valid = s0 + g < nsampled;  // groups past the end repeat the item's first token
  const uint32_t e = order[valid ? s0 + g : s0];
  const int64_t tk = t0 + (e >> kTokShift);
  const int len = (int)((e >> kLenShift) & 0xfffu);
  const int nepad = (int)(e & 0x3ffu) * 2;
  const uint2* L = p.list + tk * list_stride(p.d_in);
  const bool odd_part = cl >= HALF;
  const int part_base = odd_part ? nepad : 0;
  const int part_len = odd_part ? len - nepad : nepad;
  const int maxpart = wave_max_int(max(nepad, len - nepad));
  const uint32_t zero_row = (uint32_t)(odd_part ? zero_row_odd(p.d_in) : zero_row_even(p.d_in)) * RB;
  const int v = cl ^ ((g & 1) ? HALF : 0);
  const int h2 = 2 * (cl % HALF);
  const uint32_t lane_base = lds_addr(Ws) + (uint32_t)v * 16;  // the slice is 128-byte aligned
  float4 acc[LPR];
#pragma unroll
  for (int c = 0; c < LPR; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  // entries two rounds ahead; masked when consumed, so the loads stay in flight. Two
  // rounds per iteration, so the two buffers swap roles without register copies.
  const uint4* ep = reinterpret_cast<const uint4*>(L + part_base + h2);  // even index: 16-byte aligned
  constexpr int EPR = LPR / 2;  // entry pairs (uint4) per part per round
  uint4 n1 = ep[0], n2 = ep[EPR];
  ep += 2 * EPR;
  for (int q0 = 0; q0 < maxpart; q0 += 2 * LPR) {
    uint4 en = entry_mask(n1, q0 + h2 < part_len, zero_row);
    n1 = ep[0];
    __builtin_amdgcn_sched_barrier(0);  // keep the load two rounds ahead of its use
    row_fma<LPR>(acc, lane_base + en.x, __uint_as_float(en.y));
    row_fma<LPR>(acc, lane_base + en.z, __uint_as_float(en.w));
    if (q0 + LPR >= maxpart) break;
    en = entry_mask(n2, q0 + LPR + h2 < part_len, zero_row);
    n2 = ep[EPR];
    ep += 2 * EPR;
    __builtin_amdgcn_sched_barrier(0);
    row_fma<LPR>(acc, lane_base + en.x, __uint_as_float(en.y));
    row_fma<LPR>(acc, lane_base + en.z, __uint_as_float(en.w));
  }
  // reduce-scatter: acc[c] holds chunk c ^ v; the partner v ^ m holds it in register c ^ m
#define MCA_ADDX(a, CTRL, b) make_float4(a.x + dpp_f32<CTRL>(b.x), a.y + dpp_f32<CTRL>(b.y), \
                                       a.z + dpp_f32<CTRL>(b.z), a.w + dpp_f32<CTRL>(b.w))
  if constexpr (LPR == 8) {
    // xor 4 within 8 lanes = half-row mirror (xor 7) after quad permutation xor 3
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float4 b = acc[c + 4];
      const float4 b3 = make_float4(dpp_f32<0x1B>(b.x), dpp_f32<0x1B>(b.y), dpp_f32<0x1B>(b.z), dpp_f32<0x1B>(b.w));
      acc[c] = MCA_ADDX(acc[c], 0x141, b3);
    }
  }
  acc[0] = MCA_ADDX(acc[0], 0x4E, acc[2]);  // xor 2
  acc[1] = MCA_ADDX(acc[1], 0x4E, acc[3]);
  acc[0] = MCA_ADDX(acc[0], 0xB1, acc[1]);  // xor 1
#undef MCA_ADDX
  if (valid) store_h4<BF>(p, tk * p.d_out + c0 + 4 * v, acc[0]);
}

// The block's (slice, token range). Workgroups go to the eight XCDs in turn (block b to XCD
// b mod 8). With the slices in four groups and the token ranges in two, XCD x takes slice
// group x mod 4 of range group x / 4: every block still has one slice of one range, but an
// XCD's L2 now serves the lists and saturated x rows of half the tokens (read by four XCDs
// instead of eight) and a quarter of W_v (read by two), which about halves the kernel's
// fetch from memory. Other grid shapes keep slice = b mod nslices.
__device__ __forceinline__ void gather_block_unit(const FwdParams& p, int nslices, int& slice, int& range) {
  const int b = (int)blockIdx.x;
  if (nslices % 4 == 0 && p.gather_bps % 2 == 0 && (int)gridDim.x == nslices * p.gather_bps) {
    const int x = b % 8, k = b / 8, sq = nslices / 4;
    slice = (x % 4) * sq + k % sq;
    range = (x / 4) * (p.gather_bps / 2) + k / sq;
  } else {
    slice = b % nslices;
    range = b / nslices;
  }
}

template <int BF, int WC, bool VEC, bool LDSB>
__global__ __launch_bounds__(kThreads) void k_gather(FwdParams p) {
  constexpr int RB = WC * 4;   // bytes per slice row in LDS
  constexpr int G = 64 / (RB / 16);  // sampled tokens per work item
  extern __shared__ __align__(128) unsigned char smem_raw[];
  // the slice starts 128-byte aligned (row chunks are addressed by XOR of the chunk index)
  unsigned char* smem = smem_raw + ((128u - (lds_addr(smem_raw) & 127u)) & 127u);
  const int d_in = p.d_in, d_out = p.d_out;
  const int nslices = d_out / WC;
  int slice, bis;
  gather_block_unit(p, nslices, slice, bis);
  const int c0 = slice * WC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t ntok = (int64_t)p.B * p.n;
  float* Ws = reinterpret_cast<float*>(smem);  // [d_in + 2][WC], the last two rows zero
  uint4* Bl = reinterpret_cast<uint4*>(smem + (size_t)(d_in + 2) * WC * 4);          // LDSB: [2][nks][64]
  uint32_t* order = reinterpret_cast<uint32_t*>(smem + (size_t)(d_in + 2) * WC * 4 +
                                                (LDSB ? (size_t)2 * kLdsbSteps * 1024 : 0));  // [kChunk]
  int* satl = reinterpret_cast<int*>(order + kChunk);                                // [kChunk]
  int* ctr = satl + kChunk;                                                          // [kNumCtr]
  const int stride = list_stride(d_in);

  const int64_t per_block = (ntok + p.gather_bps - 1) / p.gather_bps;
  const int64_t t_begin = (int64_t)bis * per_block, t_end = min(t_begin + per_block, ntok);
  // the first pass's r and U, loaded together with the slice
  int r_first = 0, u_first = 0;
  if (t_begin + tid < t_end) {
    r_first = p.r[t_begin + tid];
    u_first = p.ucount[t_begin + tid];
  }

  // ---- the slice of W_v, as float32, into LDS, then two zero rows: 16-byte global loads,
  // four per thread in flight. The first four are issued now and stored after the first
  // pass has classified and counted its tokens, so that the classification overlaps their
  // latency (and a block without work never stores them).
  using TW = typename Elem<BF>::T;
  constexpr int CE = BF ? 8 : 4;  // elements per 16-byte chunk
  constexpr int CPR = WC / CE;    // chunks per slice row
  const TW* Wg = static_cast<const TW*>(p.W);
  const int nchunk = d_in * CPR;
  uint4 su[4];
#define MCA_SLICE_LOAD(V0)                                                                     \
  _Pragma("unroll") for (int h = 0; h < 4; ++h) {                                            \
    const int v = min((V0) + h * kThreads, nchunk - 1); /* clamped: stored only if in range */ \
    su[h] = *reinterpret_cast<const uint4*>(Wg + (int64_t)(v / CPR) * d_out + c0 + (v % CPR) * CE); \
  }
#define MCA_SLICE_STORE(V0)                                                                    \
  _Pragma("unroll") for (int h = 0; h < 4; ++h) {                                            \
    const int v = (V0) + h * kThreads;                                                         \
    if (v < nchunk) {                                                                          \
      float* dst = Ws + (v / CPR) * WC + (v % CPR) * CE;                                       \
      if constexpr (BF) {                                                                      \
        reinterpret_cast<float4*>(dst)[0] =                                                    \
            make_float4(__uint_as_float(su[h].x << 16), __uint_as_float(su[h].x & 0xffff0000u), \
                        __uint_as_float(su[h].y << 16), __uint_as_float(su[h].y & 0xffff0000u)); \
        reinterpret_cast<float4*>(dst)[1] =                                                    \
            make_float4(__uint_as_float(su[h].z << 16), __uint_as_float(su[h].z & 0xffff0000u), \
                        __uint_as_float(su[h].w << 16), __uint_as_float(su[h].w & 0xffff0000u)); \
      } else {                                                                                 \
        *reinterpret_cast<float4*>(dst) = make_float4(__uint_as_float(su[h].x), __uint_as_float(su[h].y), \
                                                      __uint_as_float(su[h].z), __uint_as_float(su[h].w)); \
      }                                                                                        \
    }                                                                                          \
  }
  MCA_SLICE_LOAD(tid)
  // LDSB: the slice's B fragments (2 tiles x nks steps x 1 KB, contiguous in the prepared
  // weights), at most 3 16-byte chunks per thread
  const int nfrag = LDSB ? 2 * (p.din_pad / 32) * 64 : 1;
  uint4 fu0, fu1, fu2;
  if constexpr (LDSB) {
    const uint4* src = static_cast<const uint4*>(p.Wt) + (size_t)(c0 / 16) * (p.din_pad / 32) * 64;
    fu0 = src[min(tid, nfrag - 1)];
    fu1 = src[min(tid + kThreads, nfrag - 1)];
    fu2 = src[min(tid + 2 * kThreads, nfrag - 1)];
  }
  if (tid < 2 * WC) Ws[d_in * WC + tid] = 0.f;

  // ---- classify a pass's tokens (one per thread) and sort the sampled ones by key
  int key, rank;
  uint32_t ent;
#define MCA_CLASSIFY(T0, RV, UV)                                                                \
  {                                                                                            \
    const int m = (int)min((int64_t)kChunk, t_end - (T0));                                     \
    key = -1;                                                                                  \
    rank = 0;                                                                                  \
    ent = 0;                                                                                   \
    if (tid < m) {                                                                             \
      const int r = (RV), uc = (UV);                                                           \
      const int len = min(uc & 0xffff, stride);                                                \
      const int nepad = min(min((uc >> 16) & 0xffff, len), 2046) & ~1;                         \
      if (exact_token(r, d_in, p.exact_from)) {                                                \
        if (!p.sat_separate) satl[atomicAdd(ctr, 1)] = tid;                                    \
      } else if (r > 0 && len > 0) {                                                           \
        key = sort_key(max(nepad, len - nepad));                                               \
        rank = atomicAdd(ctr + 2 + key, 1);                                                    \
        ent = ((uint32_t)tid << kTokShift) | ((uint32_t)len << kLenShift) | (uint32_t)(nepad >> 1); \
      }                                                                                        \
    }                                                                                          \
  }
  if (tid < kNumCtr) ctr[tid] = 0;
  __syncthreads();  // the counters are clear
  MCA_CLASSIFY(t_begin, r_first, u_first)

  // the classified pass's key offsets: every key's first slot in the order, longest first
  auto offsets = [&]() {
    __syncthreads();
    if (tid < 64) {  // one wave; lane l: keys 95 - 2l, 94 - 2l
      static_assert(kNumKeys == 96, "two keys per lane of one wave");
      const int kh = kNumKeys - 1 - 2 * tid, kl = kh - 1;
      const int ch = kl >= 0 ? ctr[2 + kh] : 0, cl = kl >= 0 ? ctr[2 + kl] : 0;
      const int incl = (int)wave_inclusive_scan<uint32_t>((uint32_t)(ch + cl));
      if (kl >= 0) {
        ctr[kCtrOff + kh] = incl - ch - cl;
        ctr[kCtrOff + kl] = incl - cl;
      }
      if (tid == 63) ctr[kCtrOff + kNumKeys] = incl;
    }
    __syncthreads();
  };
  if constexpr (!LDSB) {
    // saturated tokens go to their own kernel: a block whose tokens fit one pass and make no
    // work item (every token saturated, or without draws) has nothing to write and stops
    // before filling the slice (block-uniform: every thread reads the same counts). With
    // LDSB the saturated tokens are encoded here and a block almost always has work.
    offsets();
    if (ctr[0] == 0 && ctr[kCtrOff + kNumKeys] == 0 && t_begin + kChunk >= t_end) return;
  }
  // the slice into LDS (its first loads were issued before the classification), published
  // by the barrier after the first pass's order
  MCA_SLICE_STORE(tid)
  if constexpr (LDSB) {
    if (tid < nfrag) Bl[tid] = fu0;
    if (tid + kThreads < nfrag) Bl[tid + kThreads] = fu1;
    if (tid + 2 * kThreads < nfrag) Bl[tid + 2 * kThreads] = fu2;
  }
  for (int v0 = tid + 4 * kThreads; v0 < nchunk; v0 += 4 * kThreads) {
    MCA_SLICE_LOAD(v0)
    MCA_SLICE_STORE(v0)
  }

  for (int64_t t0 = t_begin;;) {
    if (LDSB || t0 != t_begin) offsets();  // block-uniform
    if (key >= 0) order[ctr[kCtrOff + key] + rank] = ent;
    __syncthreads();
    const int nsat = ctr[0];
    const int nsampled = ctr[kCtrOff + kNumKeys];
    const int ngroups = (nsat + 15) / 16;
    const int nitems = ngroups + (nsampled + G - 1) / G;
    // the next pass's r and U, loaded now so that their latency passes under this pass's items
    int r_next = 0, u_next = 0;
    if (t0 + kChunk + tid < t_end) {
      r_next = p.r[t0 + kChunk + tid];
      u_next = p.ucount[t0 + kChunk + tid];
    }

    // ---- work items from the block's queue
    for (;;) {
      int it = 0;
      if (lane == 0) it = atomicAdd(ctr + 1, 1);
      it = __builtin_amdgcn_readfirstlane(it);
      if (it >= nitems) break;
      if (it < ngroups) {
        if constexpr (LDSB) saturated_group_ldsb(p, satl, t0, it, nsat, c0, lane, Bl);
        else saturated_group<BF, WC, VEC>(p, satl, t0, it, nsat, c0, lane);
      }
      else sampled_item<BF, RB>(p, Ws, order, (it - ngroups) * G, nsampled, t0, c0, lane);
    }
    __syncthreads();  // the order and the counters are rewritten next
    t0 += kChunk;
    if (t0 >= t_end) break;
    if (tid < kNumCtr) ctr[tid] = 0;
    __syncthreads();
    MCA_CLASSIFY(t0, r_next, u_next)
  }
#undef MCA_CLASSIFY
#undef MCA_SLICE_LOAD
#undef MCA_SLICE_STORE
}

// ------------------------------------------------------------------ saturated tokens
// Exact encoding x_j W_v of the saturated tokens (r_j = d_in) as a kernel of its own, for
// the shapes where the gather cannot hold the B operand in LDS (d_in > 768, float32, or x
// rows not in 16-byte chunks). A block takes 64 consecutive tokens, lists its saturated
// tokens in LDS and multiplies them with a block of columns; each of its four waves
// computes 32 of them (two 16-row tiles). A is the x rows (k-contiguous), B the prepared
// W_v^T in fragment order (one coalesced 1 KB block per 16-column tile and k step). Every
// output row depends on its own x row only, so a token's H~ does not depend on where the
// list puts it.
//
// k_saturated (x rows not in 16-byte chunks): 128 columns per block, 64 per wave, operands
// straight from memory into registers, two k steps per round, the next round's loads
// issued before this round's MFMAs.
constexpr int kSatTokens = 64;   // tokens per block
constexpr int kSatCols = 128;    // columns per block
constexpr int kSatThreads = 256;

// The block's unit of the (token tile, column block) grid, column blocks fastest. Workgroups
// go to the eight XCDs in turn (block b to XCD b mod 8), so units are dealt out in one
// contiguous run per XCD: the column blocks of a token tile then share that XCD's L2 and
// its x rows are fetched from memory once rather than by several XCDs. A bijection of
// [0, gridDim.x).
__device__ __forceinline__ int xcd_run_unit() {
  const int nb = (int)gridDim.x, per = nb / 8, extra = nb % 8;
  const int x = (int)blockIdx.x % 8, k = (int)blockIdx.x / 8;
  return x * per + min(x, extra) + k;
}

template <int BF, bool VEC>
__global__ __launch_bounds__(kSatThreads) void k_saturated(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int E = BF ? 8 : 4;     // elements per 16 bytes
  constexpr int KS = BF ? 32 : 16;  // k per step
  constexpr int RD = 2;             // steps per round
  __shared__ int satl[kSatTokens];
  __shared__ int nsat_s;
  const int ncb = p.d_out / kSatCols;
  const int u = xcd_run_unit();
  const int cb = u % ncb, tb = u / ncb;
  const int64_t t0 = (int64_t)tb * kSatTokens;
  const int64_t ntok = (int64_t)p.B * p.n;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in;
  if (tid == 0) nsat_s = 0;
  __syncthreads();
  if (tid < kSatTokens && t0 + tid < ntok && exact_token(p.r[t0 + tid], d_in, p.exact_from))
    satl[atomicAdd(&nsat_s, 1)] = tid;
  __syncthreads();
  const int nsat = nsat_s;
  const int wm = wave >> 1, wn = wave & 1;
  if (32 * wm >= nsat) return;  // no token for this wave (wave-uniform)
  const int c0 = cb * kSatCols + 64 * wn;
  // A rows: list rows 32 wm + 16 mt + r16 (rows past the list repeat a token, not stored)
  const T* xr[2];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
    xr[mt] = static_cast<const T*>(p.X) + (t0 + satl[min(32 * wm + 16 * mt + r16, nsat - 1)]) * d_in;
  const int nks = p.din_pad / KS;
  const T* wt = static_cast<const T*>(p.Wt) + ((int64_t)(c0 / 16) * nks * 64 + lane) * E;
  f32x4_t acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nrounds = nks / RD;  // even: nks is a multiple of 4
  uint4 a0[RD][2], b0[RD][4], a1[RD][2], b1[RD][4];
#define MCA_SAT_LOAD(A, Bv, RND)                                                               \
  _Pragma("unroll") for (int u = 0; u < RD; ++u) {                                             \
    const int ks = (RND) * RD + u;                                                             \
    _Pragma("unroll") for (int mt = 0; mt < 2; ++mt) A[u][mt] = load_x_chunk<BF, VEC>(xr[mt], ks * KS + E * g, d_in); \
    _Pragma("unroll") for (int nt = 0; nt < 4; ++nt)                                           \
      Bv[u][nt] = *reinterpret_cast<const uint4*>(wt + ((int64_t)nt * nks + ks) * 64 * E);      \
  }
#define MCA_SAT_MFMA(A, Bv)                                                                    \
  _Pragma("unroll") for (int u = 0; u < RD; ++u) {                                             \
    _Pragma("unroll") for (int mt = 0; mt < 2; ++mt) {                                         \
      _Pragma("unroll") for (int nt = 0; nt < 4; ++nt) {                                       \
        if constexpr (BF) {                                                                    \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A[u][mt]), \
                                                               __builtin_bit_cast(bf16x8_t, Bv[u][nt]), \
                                                               acc[mt][nt], 0, 0, 0);          \
        } else {                                                                               \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u][mt].x), __uint_as_float(Bv[u][nt].x), acc[mt][nt], 0, 0, 0); \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u][mt].y), __uint_as_float(Bv[u][nt].y), acc[mt][nt], 0, 0, 0); \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u][mt].z), __uint_as_float(Bv[u][nt].z), acc[mt][nt], 0, 0, 0); \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[u][mt].w), __uint_as_float(Bv[u][nt].w), acc[mt][nt], 0, 0, 0); \
        }                                                                                      \
      }                                                                                        \
    }                                                                                          \
  }
  MCA_SAT_LOAD(a0, b0, 0)
  for (int rd = 0; rd < nrounds; rd += 2) {
    MCA_SAT_LOAD(a1, b1, rd + 1)
    __builtin_amdgcn_sched_barrier(0);  // the next round's loads stay ahead of these MFMAs
    MCA_SAT_MFMA(a0, b0)
    MCA_SAT_LOAD(a0, b0, min(rd + 2, nrounds - 1))
    __builtin_amdgcn_sched_barrier(0);
    MCA_SAT_MFMA(a1, b1)
  }
#undef MCA_SAT_LOAD
#undef MCA_SAT_MFMA
  // acc[mt][nt][i] = H~[list row 32 wm + 16 mt + 4 g + i][c0 + 16 nt + r16]
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 32 * wm + 16 * mt + 4 * g + i;
      if (row < nsat) {
        const int64_t base = (t0 + satl[row]) * p.d_out + c0 + r16;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) store_h<BF>(p, base + 16 * nt, acc[mt][nt][i]);
      }
    }
}

// k_saturated_lds (16-byte x chunks): 16 WN NTW columns and 32 MTW tokens per block, 2 x WN
// waves of 16 MTW tokens x 16 NTW columns each, the operands staged through LDS by direct
// global-to-LDS loads (16 bytes per lane, no registers) with ST - 1 k steps in flight. Per k
// step the block stages its 2 MTW 16-row A tiles and WN NTW 16-column B tiles in fragment
// order (1 KB each; lane l's 16 bytes at 16 l), and every wave reads its MTW A and NTW B
// fragments from there. bfloat16: 128 x 256 tiles in eight waves (MTW = NTW = 4, WN = 4),
// two per SIMD, so that one wave's LDS reads and waits pass under the other's MFMAs (eight
// fragment reads feed 16 MFMAs); float32: 64 x 256 tiles in four waves (MTW = 2, NTW = 8,
// WN = 2: ten fragment reads feed 16). A chunk past the end of a row re-reads the row's
// last chunk: the prepared W_v^T is zero there.
constexpr int kSatStages = 3;

// s_waitcnt for at most n outstanding vector memory operations (gfx9 encoding: vmcnt in
// bits 3:0 and 15:14; expcnt and lgkmcnt left at their maxima, i.e. not waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// One direct global-to-LDS load of 16 bytes per lane: lane l's bytes land at lds + 16 l
// (lds wave-uniform, in M0: an input operand bound to that register, so the compiler sets
// it and knows it is read). Issued through inline assembly so that the compiler does not
// track it: the kernel waits for these loads itself (s_waitcnt vmcnt with the count of
// loads issued after the one it needs) and publishes them with a barrier.
__device__ __forceinline__ void load_lds16(const void* g, uint32_t lds) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}

// Block barrier without a memory fence: LDS written by the direct loads is published by the
// explicit wait before it, and the compiler may not move memory operations across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int BF, int NTW, int MTW, int ST, int WN = 2>
__global__ __launch_bounds__(128 * WN) void k_saturated_lds(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int E = BF ? 8 : 4;     // elements per 16 bytes
  constexpr int KS = BF ? 32 : 16;  // k per step
  constexpr int WV = 2 * WN;        // waves: 2 along the tokens x WN along the columns
  constexpr int NA = 2 * MTW;       // A tiles per block (16 tokens each)
  constexpr int NB = WN * NTW;      // B tiles per block (16 columns each)
  constexpr int TOK = 16 * NA;      // tokens per block
  constexpr int COLS = 16 * NB;     // columns per block
  constexpr int TILES = NA + NB;    // 1 KB tiles per step slot: the A tiles, then the B tiles
  static_assert(NA % WV == 0 && NB % WV == 0, "every wave loads the same number of tiles");
  static_assert(ST >= 2, "stages");
  constexpr int kLoads = (NA + NB) / WV;  // direct loads per wave per step
  constexpr int kSlot = TILES * 64 * 16;
  __shared__ int satl[TOK];
  __shared__ int nsat_s;
  __shared__ __align__(16) uint4 stage[ST * TILES * 64];
  const int ncb = p.d_out / COLS;
  const int u = xcd_run_unit();
  const int cb = u % ncb, tb = u / ncb;
  const int64_t t0 = (int64_t)tb * TOK;
  const int64_t ntok = (int64_t)p.B * p.n;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int d_in = p.d_in;
  if (tid == 0) nsat_s = 0;
  __syncthreads();
  for (int i = tid; i < TOK; i += 64 * WV)
    if (t0 + i < ntok && exact_token(p.r[t0 + i], d_in, p.exact_from)) satl[atomicAdd(&nsat_s, 1)] = i;
  __syncthreads();
  const int nsat = nsat_s;
  if (nsat == 0) return;  // block-uniform
  const int nks = p.din_pad / KS;
  // this wave's loads: A tiles (NA / WV) wave + j (list rows 16 tile + r16, chunk E g of the
  // step) and B tiles (NB / WV) wave + j of the block's columns
  const T* xrow[NA / WV];
#pragma unroll
  for (int j = 0; j < NA / WV; ++j)
    xrow[j] = static_cast<const T*>(p.X) + (t0 + satl[min(16 * ((NA / WV) * wave + j) + r16, nsat - 1)]) * d_in;
  const int klast = d_in - E;  // last chunk of a row
  const T* wt = static_cast<const T*>(p.Wt) + ((int64_t)(cb * COLS / 16) * nks * 64 + lane) * E;
  const uint32_t st0 = lds_addr(stage);
  auto issue = [&](int ks) {
    const uint32_t slot = st0 + (uint32_t)(ks % ST) * kSlot;
#pragma unroll
    for (int j = 0; j < NA / WV; ++j)
      load_lds16(xrow[j] + min(ks * KS + E * g, klast), slot + (uint32_t)((NA / WV) * wave + j) * 1024u);
#pragma unroll
    for (int j = 0; j < NB / WV; ++j) {
      const int nt = (NB / WV) * wave + j;
      load_lds16(wt + ((int64_t)nt * nks + ks) * 64 * E, slot + (uint32_t)(NA + nt) * 1024u);
    }
  };
  const int wm = wave / WN, wn = wave % WN;
  const bool active = 16 * MTW * wm < nsat;  // wave-uniform
  f32x4_t acc[MTW][NTW];
#pragma unroll
  for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < ST - 1; ++ks) issue(min(ks, nks - 1));
  for (int ks = 0; ks < nks; ++ks) {
    wait_vmcnt<(ST - 2) * kLoads>();   // this wave's loads of step ks have landed
    stage_barrier();                    // everyone's; and step ks - 1's slot is free
    issue(min(ks + ST - 1, nks - 1));  // past the end: reloads of the last step into a free slot
    if (active) {
      const uint4* st = stage + (ks % ST) * TILES * 64;
      uint4 a[MTW], b[NTW];
#pragma unroll
      for (int mt = 0; mt < MTW; ++mt) a[mt] = st[(MTW * wm + mt) * 64 + lane];
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) b[nt] = st[(NA + NTW * wn + nt) * 64 + lane];
#pragma unroll
      for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
          if constexpr (BF) {
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[mt]),
                                                                 __builtin_bit_cast(bf16x8_t, b[nt]), acc[mt][nt], 0, 0, 0);
          } else {
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[mt].x), __uint_as_float(b[nt].x), acc[mt][nt], 0, 0, 0);
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[mt].y), __uint_as_float(b[nt].y), acc[mt][nt], 0, 0, 0);
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[mt].z), __uint_as_float(b[nt].z), acc[mt][nt], 0, 0, 0);
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[mt].w), __uint_as_float(b[nt].w), acc[mt][nt], 0, 0, 0);
          }
        }
    }
  }
  wait_vmcnt<0>();  // the trailing reloads have landed before the wave ends
  if (!active) return;
  const int c0 = cb * COLS + 16 * NTW * wn;
  // acc[mt][nt][i] = H~[list row 16 MTW wm + 16 mt + 4 g + i][c0 + 16 nt + r16]
#pragma unroll
  for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 16 * MTW * wm + 16 * mt + 4 * g + i;
      if (row < nsat) {
        const int64_t base = (t0 + satl[row]) * p.d_out + c0 + r16;
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) store_h<BF>(p, base + 16 * nt, acc[mt][nt][i]);
      }
    }
}

// Per-device host caches below are atomics: concurrent host threads may fill them at once
// (each writes the same value), and a reader sees either 0 (not yet known) or that value.
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_acquire);
  if (!n) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_release);
  }
  return n;
}

template <int BF, int WC, bool VEC, bool LDSB>
hipError_t launch_wc(const FwdParams& p, hipStream_t s) {
  const size_t lds = gather_lds_bytes(p.d_in, WC, LDSB);
  if (lds > 160 * 1024) return hipErrorInvalidValue;  // gfx950: 160 KB of LDS per workgroup
  if (LDSB && p.din_pad > 32 * kLdsbSteps) return hipErrorInvalidValue;
  // the largest slice of the variant plus the lists; allowed once per device
  static std::atomic<int> allowed[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (!allowed[dev].load(std::memory_order_acquire)) {
    // idempotent: threads racing here all set the same attribute before any of them launches
    const int dmax = LDSB ? 32 * kLdsbSteps : (WC == 32 ? 1024 : 2048);
    const hipError_t e = hipFuncSetAttribute((const void*)k_gather<BF, WC, VEC, LDSB>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)gather_lds_bytes(dmax, WC, LDSB));
    if (e != hipSuccess) return e;
    allowed[dev].store(1, std::memory_order_release);
  }
  const int nslices = p.d_out / WC;
  return launch_stage_kernel(k_gather<BF, WC, VEC, LDSB>, dim3((unsigned)(nslices * p.gather_bps)), dim3(kThreads),
                             lds, s, p);
}

}  // namespace

// Blocks per slice: every block gets a CU of its own (a block holds most of a CU's LDS).
int gather_blocks_per_slice(int d_in, int d_out) {
  const int nslices = d_out / gather_slice_cols(d_in);
  return max(1, device_cus() / nslices);
}

hipError_t launch_saturated(const FwdParams& p, hipStream_t s) {
  if (p.d_out % kSatCols != 0) return hipErrorInvalidValue;
  const bool vec = p.d_in % (p.bf16 ? 8 : 4) == 0;
  const int64_t ntok = (int64_t)p.B * p.n;
  const dim3 grid((unsigned)(((ntok + kSatTokens - 1) / kSatTokens) * (p.d_out / kSatCols))), blk(kSatThreads);
  if (vec && p.d_out % 256 == 0) {  // 128 (bf16) or 64 (float32) tokens x 256 columns per block
    const int tok = p.bf16 ? 128 : 64;
    const dim3 g2((unsigned)(((ntok + tok - 1) / tok) * (p.d_out / 256)));
    return p.bf16 ? launch_stage_kernel(k_saturated_lds<1, 4, 4, kSatStages, 4>, g2, dim3(512), 0, s, p)
                  : launch_stage_kernel(k_saturated_lds<0, 8, 2, kSatStages, 2>, g2, dim3(256), 0, s, p);
  }
  return p.bf16 ? launch_stage_kernel(k_saturated<1, false>, grid, blk, 0, s, p)
                : launch_stage_kernel(k_saturated<0, false>, grid, blk, 0, s, p);
}

hipError_t launch_gather(const FwdParams& p, hipStream_t s) {
  if (p.wc != gather_slice_cols(p.d_in) || p.d_out % p.wc != 0 || p.gather_bps < 1) return hipErrorInvalidValue;
  const bool vec = p.d_in % (p.bf16 ? 8 : 4) == 0;
  if (p.sat_separate) {
    if (p.bf16) {
      if (p.wc == 32) return vec ? launch_wc<1, 32, true, false>(p, s) : launch_wc<1, 32, false, false>(p, s);
      return vec ? launch_wc<1, 16, true, false>(p, s) : launch_wc<1, 16, false, false>(p, s);
    }
  }
  if (p.bf16) {
    if (p.wc == 32) {
      // bfloat16, d_in <= 768: the saturated tokens' B operand fits in LDS next to the slice
      if (vec && p.din_pad <= 32 * kLdsbSteps) return launch_wc<1, 32, true, true>(p, s);
      return vec ? launch_wc<1, 32, true, false>(p, s) : launch_wc<1, 32, false, false>(p, s);
    }
    return vec ? launch_wc<1, 16, true, false>(p, s) : launch_wc<1, 16, false, false>(p, s);
  }
  if (p.wc == 32) return vec ? launch_wc<0, 32, true, false>(p, s) : launch_wc<0, 32, false, false>(p, s);
  return vec ? launch_wc<0, 16, true, false>(p, s) : launch_wc<0, 16, false, false>(p, s);
}

}  // namespace mca
