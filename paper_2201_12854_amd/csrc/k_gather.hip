// Value encoding of the MCA forward pass on gfx950: H~[j] for every token that is not
// padded or zero, one column slice of W_v per block.
//
//   sampled token (0 < r_j < d_in): H~[j] = sum over its distinct sampled rows i of
//     coef_i W_v[i, :] (Eq. 2 with duplicates merged; Eq. 5 inner sum), float32
//     accumulation;
//   saturated token (r_j = d_in): H~[j] = x_j W_v exactly, on MFMA (16 tokens per tile).
//
// The slice W_v[:, c0 .. c0 + WC) is converted to float32 once and kept in LDS for the
// whole block (768 x 32 floats = 96 KB: the 160 KB LDS of a gfx950 CU holds it), so the
// gather reads LDS instead of L2. A row of the slice is WC / 4 lanes x 16 bytes; a wave
// works on 64 / (WC / 4) sampled tokens at once, one per lane group, so each 16-byte LDS
// read instruction fetches one sampled row for each of them and no cross-lane reduction
// is needed. The list entries (LDS byte offset of the row, coefficient) are loaded one
// round ahead with coalesced 16-byte loads and shared within each lane group through a
// small LDS staging area.
//
// Work distribution: the blocks of a slice split the tokens into contiguous ranges. A block
// reads r and U of its range, puts the saturated tokens on one LDS list and sorts the
// sampled tokens by list length (key floor(4 log2 U), longest first) with LDS atomics; its
// waves then take work items from an LDS counter: groups of 16 saturated tokens first
// (the heaviest items), then groups of sampled tokens of similar length, longest first,
// so that the lanes of a wave and the waves of a block finish close together. No global
// atomics; outputs do not depend on which wave computes them.
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
  constexpr int DEPTH = 4;          // steps per round (din_pad / KS is a multiple of 4)
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
  // rounds of DEPTH steps: all loads of the round, then its MFMAs. din_pad is a multiple of
  // 128 elements, so every round is whole and the loop has no conditional code (the
  // padded k carry zero weights; x past d_in reads as zero).
  for (int ks0 = 0; ks0 < nks; ks0 += DEPTH) {
    uint4 a[DEPTH], w[DEPTH][NC];
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) {
      const int ks = ks0 + u;
      a[u] = load_x_chunk<BF, VEC>(xrow, ks * KS + (BF ? 8 : 4) * g, d_in);
#pragma unroll
      for (int c = 0; c < NC; ++c)
        w[u][c] = *reinterpret_cast<const uint4*>(wt + ((int64_t)c * nks + ks) * 64 * E);
    }
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        if constexpr (BF) {
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[u]),
                                                          __builtin_bit_cast(bf16x8_t, w[u][c]), acc[c], 0, 0, 0);
        } else {
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[u].x), __uint_as_float(w[u][c].x), acc[c], 0, 0, 0);
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[u].y), __uint_as_float(w[u][c].y), acc[c], 0, 0, 0);
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[u].z), __uint_as_float(w[u][c].z), acc[c], 0, 0, 0);
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[u].w), __uint_as_float(w[u][c].w), acc[c], 0, 0, 0);
        }
      }
    }
  }
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

// Max / min over the 64 lanes, returned in a scalar register.
__device__ __forceinline__ int wave_max_int(int v) {
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, true));
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, true));
  return max(max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}

// acc += coef * W_lds[row] (4 columns) for one list entry (LDS byte offset of the row, coef).
__device__ __forceinline__ void fma_row(float4& acc, const unsigned char* wl, uint2 e) {
  const float4 w = *reinterpret_cast<const float4*>(wl + e.x);
  const float c = __uint_as_float(e.y);
  acc.x = fmaf(c, w.x, acc.x);
  acc.y = fmaf(c, w.y, acc.y);
  acc.z = fmaf(c, w.z, acc.z);
  acc.w = fmaf(c, w.w, acc.w);
}

constexpr int kChunk = kThreads;  // tokens classified per block pass (one per thread)
constexpr int kNumKeys = 48;      // sort keys floor(4 log2 U) for 1 <= U < 4096
constexpr int kUBits = 12;        // order entry: (local token << 12) | U

// floor(4 log2 U) for 1 <= U < 4096: the octave and the next two bits of U.
__device__ __forceinline__ int sort_key(int U) {
  const int e = 31 - __clz(U);
  const int f = e >= 2 ? (U >> (e - 2)) & 3 : (U << (2 - e)) & 3;
  return 4 * e + f;
}

constexpr int kWavesPerBlock = kThreads / 64;

__host__ __device__ inline size_t gather_lds_bytes(int d_in, int wc) {
  return (size_t)(d_in + 1) * wc * 4         // W_v slice, float32, and a zero row
         + (size_t)kWavesPerBlock * 1024      // list staging, 1 KB per wave
         + (size_t)kChunk * 4 * 2            // sampled order, saturated list
         + 64 * 4;                           // counters
}

// Orders LDS accesses of different lanes of one wavefront: the hardware executes a wave's
// LDS instructions in issue order, so only compiler reordering has to be prevented.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// This lane's two list entries q, q + 1 (q even, 16 bytes) of a list of length U; entries
// past the end become the zero row with coefficient 0. The load address is clamped into
// the token's list slot (stride entries, even) and the selection done with masks, so the
// load needs no branch.
__device__ __forceinline__ uint4 entry_pair(const uint2* L, int q, int U, int stride, uint32_t zero_row) {
  const uint4 v = *reinterpret_cast<const uint4*>(L + min(q, stride - 2));
  const uint32_t k0 = q < U ? 0xffffffffu : 0u, k1 = q + 1 < U ? 0xffffffffu : 0u;
  return make_uint4((v.x & k0) | (zero_row & ~k0), v.y & k0, (v.z & k1) | (zero_row & ~k1), v.w & k1);
}

// G = 64 / (RB / 16) sampled tokens s0 .. s0 + G - 1 of the sorted order, one per lane group:
// group g accumulates its token's rows for the 4 columns 4 cl .. 4 cl + 3 of every lane.
// A round covers RB / 8 list entries of every group: the wave loads them with one
// coalesced 16-byte load per lane (lane cl of group g: entries 2 cl, 2 cl + 1 of its
// token), one round ahead, writes them to its LDS staging area and every group reads its
// own entries back as broadcast reads. A wave's LDS instructions execute in issue order,
// so one staging buffer per wave suffices.
template <int BF, int RB>
__device__ void sampled_item(const FwdParams& p, const float* Ws, uint4* stage, const uint32_t* order, int s0,
                             int nsampled, int64_t t0, int c0, int lane) {
  constexpr int LPR = RB / 16;    // lanes per row and per group
  constexpr int NE = 2 * LPR;     // entries per group per round
  const int g = lane / LPR, cl = lane % LPR;
  const bool valid = s0 + g < nsampled;  // groups past the end repeat the item's first token
  const uint32_t e = order[valid ? s0 + g : s0];
  const int64_t tk = t0 + (e >> kUBits);
  const int U = (int)(e & ((1u << kUBits) - 1u));  // >= 1
  const int stride = list_stride(p.d_in);
  const uint2* L = p.list + tk * stride;
  const int maxU = wave_max_int(U);
  const uint32_t zero_row = (uint32_t)p.d_in * RB;
  const unsigned char* wl = reinterpret_cast<const unsigned char*>(Ws) + cl * 16;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  uint4 nxt = entry_pair(L, 2 * cl, U, stride, zero_row);
  for (int q0 = 0; q0 < maxU; q0 += NE) {
    uint4* st = stage;
    wave_lds_sync();  // the previous round's reads stay ahead of this write
    st[lane] = nxt;
    wave_lds_sync();
    nxt = entry_pair(L, q0 + NE + 2 * cl, U, stride, zero_row);  // next round (unused after the last)
    const uint4* mine = st + g * LPR;                      // this group's NE entries
    // all entry reads, then all row reads (distinct registers, so they are in flight
    // together), then the FMAs
    uint4 two[LPR];
#pragma unroll
    for (int k = 0; k < LPR; ++k) two[k] = mine[k];
    float4 w[2 * LPR];
#pragma unroll
    for (int k = 0; k < LPR; ++k) {
      w[2 * k] = *reinterpret_cast<const float4*>(wl + two[k].x);
      w[2 * k + 1] = *reinterpret_cast<const float4*>(wl + two[k].z);
    }
#pragma unroll
    for (int k = 0; k < 2 * LPR; ++k) {
      const float c = __uint_as_float((k & 1) ? two[k >> 1].w : two[k >> 1].y);
      acc.x = fmaf(c, w[k].x, acc.x);
      acc.y = fmaf(c, w[k].y, acc.y);
      acc.z = fmaf(c, w[k].z, acc.z);
      acc.w = fmaf(c, w[k].w, acc.w);
    }
  }
  if (valid) store_h4<BF>(p, tk * p.d_out + c0 + 4 * cl, acc);
}

template <int BF, int WC, bool VEC>
__global__ __launch_bounds__(kThreads) void k_gather(FwdParams p) {
  constexpr int RB = WC * 4;   // bytes per slice row in LDS
  constexpr int G = 64 / (RB / 16);  // sampled tokens per work item
  extern __shared__ __align__(16) unsigned char smem[];
  const int d_in = p.d_in, d_out = p.d_out;
  const int nslices = d_out / WC;
  const int slice = blockIdx.x % nslices, bis = blockIdx.x / nslices;
  const int c0 = slice * WC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t ntok = (int64_t)p.B * p.n;
  float* Ws = reinterpret_cast<float*>(smem);  // [d_in + 1][WC], the last row zero
  uint4* stage = reinterpret_cast<uint4*>(smem + (size_t)(d_in + 1) * WC * 4) + (tid >> 6) * 64;  // 64 per wave
  uint32_t* order = reinterpret_cast<uint32_t*>(smem + (size_t)(d_in + 1) * WC * 4 + kWavesPerBlock * 1024);
  int* satl = reinterpret_cast<int*>(order + kChunk);                                // [kChunk]
  int* ctr = satl + kChunk;  // [0] saturated, [1 + key] sort-key counts, [60] work queue

  const int64_t per_block = (ntok + p.gather_bps - 1) / p.gather_bps;
  const int64_t t_begin = (int64_t)bis * per_block, t_end = min(t_begin + per_block, ntok);
  // the first pass's r and U, loaded together with the slice
  int r_first = 0, u_first = 0;
  if (t_begin + tid < t_end) {
    r_first = p.r[t_begin + tid];
    u_first = p.ucount[t_begin + tid];
  }

  // ---- the slice of W_v, as float32, into LDS, then a zero row: 16-byte global loads,
  // four per thread in flight before the conversions and LDS stores
  if (tid < WC) Ws[d_in * WC + tid] = 0.f;
  {
    using T = typename Elem<BF>::T;
    constexpr int CE = BF ? 8 : 4;  // elements per 16-byte chunk
    constexpr int CPR = WC / CE;    // chunks per slice row
    const T* W = static_cast<const T*>(p.W);
    const int nchunk = d_in * CPR;
    for (int v0 = tid; v0 < nchunk; v0 += 4 * kThreads) {
      uint4 u[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int v = min(v0 + h * kThreads, nchunk - 1);  // clamped: in range, stored only if v < nchunk
        u[h] = *reinterpret_cast<const uint4*>(W + (int64_t)(v / CPR) * d_out + c0 + (v % CPR) * CE);
      }
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int v = v0 + h * kThreads;
        if (v < nchunk) {
          float* dst = Ws + (v / CPR) * WC + (v % CPR) * CE;
          if constexpr (BF) {
            reinterpret_cast<float4*>(dst)[0] =
                make_float4(__uint_as_float(u[h].x << 16), __uint_as_float(u[h].x & 0xffff0000u),
                            __uint_as_float(u[h].y << 16), __uint_as_float(u[h].y & 0xffff0000u));
            reinterpret_cast<float4*>(dst)[1] =
                make_float4(__uint_as_float(u[h].z << 16), __uint_as_float(u[h].z & 0xffff0000u),
                            __uint_as_float(u[h].w << 16), __uint_as_float(u[h].w & 0xffff0000u));
          } else {
            *reinterpret_cast<float4*>(dst) = make_float4(__uint_as_float(u[h].x), __uint_as_float(u[h].y),
                                                          __uint_as_float(u[h].z), __uint_as_float(u[h].w));
          }
        }
      }
    }
  }

  for (int64_t t0 = t_begin; t0 < t_end; t0 += kChunk) {
    const int m = (int)min((int64_t)kChunk, t_end - t0);
    if (tid < 64) ctr[tid] = 0;
    __syncthreads();  // also: the slice is in LDS, the previous pass is done
    // ---- classify this pass's tokens (one per thread) and sort the sampled ones by key
    int key = -1, rank = 0, U = 0;
    if (tid < m) {
      const int r = t0 == t_begin ? r_first : p.r[t0 + tid];
      U = min(max(t0 == t_begin ? u_first : p.ucount[t0 + tid], 0), d_in);
      if (r >= d_in) {
        satl[atomicAdd(ctr, 1)] = tid;
      } else if (r > 0 && U > 0) {
        key = sort_key(U);
        rank = atomicAdd(ctr + 1 + key, 1);
      }
    }
    __syncthreads();
    if (key >= 0) {
      int off = 0;  // longer lists first
      for (int k = kNumKeys - 1; k > key; --k) off += ctr[1 + k];
      order[off + rank] = ((uint32_t)tid << kUBits) | (uint32_t)U;
    }
    __syncthreads();
    const int nsat = ctr[0];
    int nsampled = 0;
    for (int k = 0; k < kNumKeys; ++k) nsampled += ctr[1 + k];
    const int ngroups = (nsat + 15) / 16;
    const int nitems = ngroups + (nsampled + G - 1) / G;

    // ---- work items from the block's queue
    for (;;) {
      int it = 0;
      if (lane == 0) it = atomicAdd(ctr + 60, 1);
      it = __builtin_amdgcn_readfirstlane(it);
      if (it >= nitems) break;
      if (it < ngroups) saturated_group<BF, WC, VEC>(p, satl, t0, it, nsat, c0, lane);
      else sampled_item<BF, RB>(p, Ws, stage, order, (it - ngroups) * G, nsampled, t0, c0, lane);
    }
    __syncthreads();  // the lists of this pass are rewritten next
  }
}

int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <int BF, int WC, bool VEC>
hipError_t launch_wc(const FwdParams& p, hipStream_t s) {
  const size_t lds = gather_lds_bytes(p.d_in, WC);
  if (lds > 160 * 1024) return hipErrorInvalidValue;  // gfx950: 160 KB of LDS per workgroup
  // the largest slice (2048 x 16 or 1024 x 32 floats) plus the lists; allowed once per device
  static int allowed[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (!allowed[dev]) {
    const hipError_t e = hipFuncSetAttribute((const void*)k_gather<BF, WC, VEC>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)gather_lds_bytes(WC == 32 ? 1024 : 2048, WC));
    if (e != hipSuccess) return e;
    allowed[dev] = 1;
  }
  const int nslices = p.d_out / WC;
  hipLaunchKernelGGL((k_gather<BF, WC, VEC>), dim3((unsigned)(nslices * p.gather_bps)), dim3(kThreads), lds, s, p);
  return hipGetLastError();
}

}  // namespace

// Blocks per slice: every block gets a CU of its own (a block holds most of a CU's LDS).
int gather_blocks_per_slice(int d_in, int d_out) {
  const int nslices = d_out / gather_slice_cols(d_in);
  return max(1, device_cus() / nslices);
}

hipError_t launch_gather(const FwdParams& p, hipStream_t s) {
  if (p.wc != gather_slice_cols(p.d_in) || p.d_out % p.wc != 0 || p.gather_bps < 1) return hipErrorInvalidValue;
  const bool vec = p.d_in % (p.bf16 ? 8 : 4) == 0;
  if (p.bf16) {
    if (p.wc == 32) return vec ? launch_wc<1, 32, true>(p, s) : launch_wc<1, 32, false>(p, s);
    return vec ? launch_wc<1, 16, true>(p, s) : launch_wc<1, 16, false>(p, s);
  }
  if (p.wc == 32) return vec ? launch_wc<0, 32, true>(p, s) : launch_wc<0, 32, false>(p, s);
  return vec ? launch_wc<0, 16, true>(p, s) : launch_wc<0, 16, false>(p, s);
}

}  // namespace mca
