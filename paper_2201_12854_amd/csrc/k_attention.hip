// Attention stages of the MCA forward pass on gfx950:
//   scores + row softmax statistics + column max   (softmax(a Q K^T), a = 1/8, and the
//                                                    per-block part of max A[:, j], Eq. 8/9;
//                                                    or of the column sum (mean rule), or
//                                                    every probability (median rule))
//   Y = A H~                                        ("Y = AH", Sec. "Self-Attention
//                                                    Mechanisms"; Eq. 5 outer sum)
// Both kernels compute a probability the same way, A = exp2(fma(q . k, log2(e)/8, -c))
// with the row normaliser c written by the score pass. A is never written to memory
// (except under the median rule).
//
// Tiling: one block = 4 waves = 64 queries of one (batch row, head), a wave owning 16
// queries (the streaming kernels: 128 queries, 32 per wave in two 16-query tiles). Keys
// come in tiles of 64 staged in LDS; 16x16 MFMA tiles (bf16 16x16x32 or fp32 16x16x4).
// The score pass computes S = Q K^T (its layout and reductions are described with the
// kernels). The output pass computes S^T = K Q^T, so lane l holds the scores of query
// (l % 16) for keys 16 s + 4 (l / 16) + i (s, i = 0..3): exactly the A-operand layout of
// the P V MFMA, with no data movement between the two products.
//
// Variants by padded length:
//   resident (up to 64 NT keys, NT <= 4 for bf16, 2 for fp32): every K (and H~) tile of
//     the sequence is loaded at once behind one barrier and all scores stay in registers,
//     so the statistics and the column max come from a single pass;
//   score pass up to 8 key tiles: K tiles streamed through two LDS buffers, every score
//     kept in registers, still a single pass;
//   streaming (longer sequences): tiles are double buffered in LDS with the next tile
//     prefetched into registers; the score pass sweeps twice (per-lane statistics, then
//     the column statistic).
// Local-window attention (Sec. "Longformer": a window of w keys around each token and a
// global first token): query q attends key k < len when |q - k| <= w / 2, or q = 0, or
// k = 0; the other scores are masked like padded keys. The column max is then taken of
// |S_q| A[q, k], |S_q| the number of keys query q attends (the count rule's per-row factor
// n of Eq. 9), and the streaming variants visit only the key tiles a query tile's window
// reaches, plus tile 0 (all tiles for the tile holding query 0).
//
// Rows past the padded length are read from the last row instead of being zero-filled:
// their scores are masked and their probabilities are exactly 0. Tile loads are
// unconditional (a tile index past the last valid tile is clamped to it), which keeps the
// tiles in registers and the load stream free of divergent branches.
#include "mca_device.h"
#include "mca_kernels.h"

namespace mca {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;                // queries per block and keys per tile
// bf16 tiles in LDS: rows of 64 elements (128 bytes, no padding) whose eight 16-byte
// chunks are permuted per row, chunk c of row r stored at chunk c ^ (r & 7). gfx950 serves a
// wave's 16-byte LDS accesses in four cycles, and its transposing 8-byte reads in two, only
// when the lanes served together fall in distinct banks; with this permutation that holds
// for the three accesses to a tile (a bank-conflict probe measured each): the fragment
// reads of Q K^T (16 consecutive rows, one chunk), the transposing reads of P V (rows
// 4 g + i, one pair of chunks) and the row stores. Unpermuted 128-byte rows serialise the
// fragment reads four ways, 144-byte rows two ways.
constexpr int kStrideBf = kDHead;
// The streaming output pass keeps its H~ tiles unpermuted in 160-byte rows instead (also
// conflict-free for the transposing reads): there the four column groups of a read are
// constant offsets from one address, where the permutation would need a register per group
// and take the kernel past the register count that allows three waves per SIMD.
constexpr int kStrideBfWide = kDHead + 16;
// element offset of (row, col) in a bf16 tile; col a multiple of 4 (an 8-byte piece)
__device__ __forceinline__ int kv_at(int row, int col) {
  return row * kStrideBf + ((((col >> 3) ^ (row & 7)) << 3) | (col & 7));
}
constexpr int kStrideF = kDHead + 4;     // LDS row stride of fp32 tiles (elements)

template <int BF> struct Elem { using T = float; };
template <> struct Elem<1> { using T = uint16_t; };
template <int BF> constexpr int stride_of() { return BF ? kStrideBf : kStrideF; }

// ------------------------------------------------------------------ Q fragments
// The wave's 16 queries as the B operand of S^T = K Q^T.
template <int BF> struct QFrag;
template <> struct QFrag<1> { bf16x8_t v[2]; };   // d = 32 ks + 8 g + (0..7)
template <> struct QFrag<0> { float v[16]; };      // d = 16 g + t

__device__ __forceinline__ void load_qfrag(QFrag<1>& f, const uint16_t* qrow, int g) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
    f.v[ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * ks + 8 * g));
}

__device__ __forceinline__ void load_qfrag(QFrag<0>& f, const float* qrow, int g) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const float4 u = *reinterpret_cast<const float4*>(qrow + 16 * g + 4 * c);
    f.v[4 * c + 0] = u.x;
    f.v[4 * c + 1] = u.y;
    f.v[4 * c + 2] = u.z;
    f.v[4 * c + 3] = u.w;
  }
}

// ------------------------------------------------------------------ tiles in flight
// A 64-row x 64-column tile of a [*, d_out] matrix (the head's column slice) held in
// registers between its global load and its LDS store: 16-byte vectors v0, v1 (bf16) or
// v0..v3 (fp32) per thread; vector v of the tile is row v / R, chunk v % R (R vectors per
// row). Rows past the padded length read as zeros. (Plain members, no arrays: the tiles
// are carried across loop iterations and must stay in registers.)
struct TileRegs {
  uint4 v0, v1, v2, v3;
};

// The loads go through a buffer descriptor built per tile in scalar registers: its base is
// the tile's first row and its size ends with the head's slice of the last valid row, so
// the per-lane offset (row within the tile times the row pitch, plus the chunk) is the
// same for every tile and no per-tile address arithmetic runs on the vector units; the
// hardware range check returns zeros for rows at or past n (whose keys are masked).
constexpr int kBufWord3 = 0x00020000;  // gfx9 descriptor word 3: 32-bit data format

// The descriptor of the tile whose first row is key0: with r = min(n - key0, 64) valid rows
// its size is (r - 1) pitch + 64 elements, and 0 when r <= 0 (the pitch, d_out elements, is
// at least 256 of them, so the max() below needs no branch).
template <int BF>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void* base, int64_t ld, int key0, int n) {
  constexpr int ES = (int)sizeof(typename Elem<BF>::T);
  const int bytes = max((min(n - key0, kTile) - 1) * (int)ld * ES + kDHead * ES, 0);
  return __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(static_cast<const char*>(base) + (int64_t)key0 * ld * ES), 0, bytes, kBufWord3);
}

// vector v of the tile
template <int BF>
__device__ __forceinline__ uint4 tile_vec_load(__amdgpu_buffer_rsrc_t rs, int64_t ld, int v) {
  constexpr int R = BF ? 8 : 16;
  constexpr int ES = (int)sizeof(typename Elem<BF>::T);
  const int off = (v / R) * (int)ld * ES + (v % R) * 16;
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

template <int BF>
__device__ __forceinline__ TileRegs tile_load(const void* base, int64_t ld, int key0, int n, int tid) {
  const __amdgpu_buffer_rsrc_t rs = tile_rsrc<BF>(base, ld, key0, n);
  TileRegs t;
  t.v0 = tile_vec_load<BF>(rs, ld, tid);
  t.v1 = tile_vec_load<BF>(rs, ld, tid + kThreads);
  if constexpr (!BF) {
    t.v2 = tile_vec_load<BF>(rs, ld, tid + 2 * kThreads);
    t.v3 = tile_vec_load<BF>(rs, ld, tid + 3 * kThreads);
  } else {
    t.v2 = t.v3 = make_uint4(0, 0, 0, 0);
  }
  return t;
}

// row-major LDS tile [key][d]
template <int BF>
__device__ __forceinline__ void tile_vec_store(uint4 u, typename Elem<BF>::T* lds, int v) {
  constexpr int R = BF ? 8 : 16;
  if constexpr (BF) *reinterpret_cast<uint4*>(lds + kv_at(v / R, (v % R) * 8)) = u;
  else *reinterpret_cast<uint4*>(lds + (v / R) * kStrideF + (v % R) * 4) = u;
}

template <int BF>
__device__ __forceinline__ void tile_store(const TileRegs& t, typename Elem<BF>::T* lds, int tid) {
  tile_vec_store<BF>(t.v0, lds, tid);
  tile_vec_store<BF>(t.v1, lds, tid + kThreads);
  if constexpr (!BF) {
    tile_vec_store<BF>(t.v2, lds, tid + 2 * kThreads);
    tile_vec_store<BF>(t.v3, lds, tid + 3 * kThreads);
  }
}

// H~ tiles are stored like K tiles, row-major [key][column]; the P V MFMA reads its B
// operand (8 keys of one column per lane) with the transposing LDS read below.
template <int BF, bool WIDE = false>
__device__ __forceinline__ void tile_store_v(const TileRegs& t, typename Elem<BF>::T* lds, int tid) {
  if constexpr (BF && WIDE) {
    *reinterpret_cast<uint4*>(lds + (tid / 8) * kStrideBfWide + (tid % 8) * 8) = t.v0;
    *reinterpret_cast<uint4*>(lds + (tid / 8 + kThreads / 8) * kStrideBfWide + (tid % 8) * 8) = t.v1;
  } else {
    tile_store<BF>(t, lds, tid);
  }
}

// ds_read_b64_tr_b16 (gfx950). Within each row of 16 lanes, every lane supplies the address
// of 4 consecutive 16-bit elements; lane i receives, as its element k (k = 0..3), element
// i % 4 of the 4 addressed by lane 4 k + i / 4 of its row. Lane s addressing
// V[kb + s / 4][d0 + 4 (s % 4)] of a row-major tile therefore gives lane i the column
// V[kb .. kb + 3][d0 + i].
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

__device__ __forceinline__ uint2 lds_read_tr16(const uint16_t* p) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)p));
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
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(Ks + kv_at(16 * s + r16, 32 * ks + 8 * g));
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

// Logits in base-2 units: a (q . k) log2(e) with a = 1/sqrt(64), the rounded constant
// log2(e) / 8, so that softmax needs only exp2 (one hardware instruction):
// exp(a x - m) = exp2(a log2(e) x - m log2(e)). An attention probability is
// A = exp2(fma(dot, log2(e) / 8, -c)) with the row's c = M + log2(sum of exp2(logit - M)).
constexpr float kLog2eOver8 = (float)(1.4426950408889634 / 8.0);
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }  // exp2(-inf) = 0

// max of floats on the VALU max instructions, without the operand canonicalisation the
// compiler adds around fmaxf: v_max_f32 and the three-input v_max3_f32. The operands are
// scores, statistics and probabilities (finite or -inf), whose maximum is exact.
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

__device__ __forceinline__ int valid_len(const FwdParams& p, int b) {
  int len = p.seq_lens ? p.seq_lens[b] : p.n;
  return min(max(len, 1), p.n);
}

// P V for one 64-key tile: acc holds the probabilities (S^T layout), Vs the H~ tile.
__device__ __forceinline__ void pv_tile(f32x4_t y[4], const f32x4_t acc[4], const uint16_t* Vs, int r16, int g) {
  // 32 keys per MFMA: k-slots 0..3 = keys 32 pp + 4 g + (0..3), 4..7 = keys 32 pp + 16 + 4 g + (0..3)
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    const uint4 pa = make_uint4(pack_bf16x2(acc[2 * pp][0], acc[2 * pp][1]), pack_bf16x2(acc[2 * pp][2], acc[2 * pp][3]),
                                pack_bf16x2(acc[2 * pp + 1][0], acc[2 * pp + 1][1]),
                                pack_bf16x2(acc[2 * pp + 1][2], acc[2 * pp + 1][3]));
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, pa);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      // lane (g, r16) addresses key 32 pp + 4 g + r16 / 4, columns 16 c + 4 (r16 % 4) .. + 3
      // rows 32 pp + 4 g + r16 / 4 and 16 further (the same permutation: it depends on row & 7)
      const uint16_t* vrow = Vs + kv_at(32 * pp + 4 * g + (r16 >> 2), 16 * c + 4 * (r16 & 3));
      const uint2 lo = lds_read_tr16(vrow);
      const uint2 hi = lds_read_tr16(vrow + 16 * kStrideBf);
      const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
      y[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bv, y[c], 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void pv_tile(f32x4_t y[4], const f32x4_t acc[4], const float* Vs, int r16, int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* vrow = Vs + (16 * s + 4 * g + i) * kStrideF + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) y[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[s][i], vrow[16 * c], y[c], 0, 0, 0);
    }
}

struct BlockCtx {
  int qt, h, b, tid, wave, lane, r16, g, n, d_out, len, q, ntl;
  int half;       // local window: keys within half of the query (0: full attention)
  int tlo, thi;   // key tiles visited: 0, then tlo .. thi (tlo >= 1)
  int klo, kspan; // local window: the lane's query attends keys klo .. klo + kspan, and key 0
};

// One-dimensional grid of qtiles * H * B blocks. Consecutive blocks go to the 8 XCDs in
// turn, each with its own L2; the query tiles of one (batch row, head) read the same K
// (and H~) tile, so they are placed 8 block ids apart, on the same XCD, and the second
// read hits its L2 (when H * B is a multiple of 8; otherwise in plain order).
__device__ __forceinline__ BlockCtx block_ctx(const FwdParams& p) {
  BlockCtx c;
  const int bid = blockIdx.x, Q = p.qtiles, P = p.H * p.B;
  int pair;
  if (P % 8 == 0) {
    const int G = 8 * Q, w = bid % G;
    pair = bid / G * 8 + w % 8;
    c.qt = w / 8;
  } else {
    pair = bid / Q;
    c.qt = bid % Q;
  }
  c.h = pair % p.H;
  c.b = pair / p.H;
  c.tid = threadIdx.x;
  c.wave = c.tid >> 6;
  c.lane = c.tid & 63;
  c.r16 = c.lane & 15;
  c.g = c.lane >> 4;
  c.n = p.n;
  c.d_out = p.d_out;
  c.len = valid_len(p, c.b);
  c.q = c.qt * kTile + c.wave * 16 + c.r16;
  c.ntl = (c.len + kTile - 1) / kTile;  // tiles past the valid length are all masked
  c.half = p.band_half;
  c.tlo = 1;
  c.thi = c.ntl - 1;
  c.klo = 0;
  c.kspan = 0;
  if (c.half > 0) {  // the window cut to the valid keys; every valid key for query 0
    int lo = c.q == 0 ? 0 : max(0, c.q - c.half);
    int hi = c.q == 0 ? c.len - 1 : min(c.len - 1, c.q + c.half);
    if (hi < lo) lo = hi = 1 << 30;  // a padded query past the window's reach: key 0 only
    c.klo = lo;
    c.kspan = hi - lo;
  }
  if (c.half > 0 && c.qt > 0) {  // the window of queries q0 .. q0 + 63
    const int q0 = c.qt * kTile;
    c.tlo = max(1, max(q0 - c.half, 0) / kTile);
    c.thi = min(c.ntl - 1, (q0 + kTile - 1 + c.half) / kTile);
  }
  return c;
}

// Key tiles a block visits, in order: tile 0, then tlo .. thi.
__device__ __forceinline__ int tile_count(const BlockCtx& c) { return 1 + max(0, c.thi - c.tlo + 1); }
__device__ __forceinline__ int tile_at(const BlockCtx& c, int idx) { return idx == 0 ? 0 : c.tlo + idx - 1; }

// Key e = 16 s + 4 g + i of tile kt (lim = len - 64 kt) is attended by the lane's query:
// a valid key (full attention), or a key in klo .. klo + kspan or key 0 (local window; one
// unsigned compare per key).
template <bool BAND>
__device__ __forceinline__ bool key_ok(const BlockCtx& c, int kt, int lim, int s, int i) {
  const int e = 16 * s + 4 * c.g + i;
  if constexpr (BAND) {
    const bool in = (unsigned)(kt * kTile + e - c.klo) <= (unsigned)c.kspan;
    return (s == 0 && i == 0) ? (in || (kt == 0 && c.g == 0)) : in;
  } else {
    return lim >= kTile || e < lim;
  }
}

// The same for the output pass's probabilities (S^T layout): masked keys get 0.
template <bool BAND>
__device__ __forceinline__ void mask_tile(f32x4_t acc[4], const BlockCtx& c, int kt, int lim) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (!key_ok<BAND>(c, kt, lim, s, i)) acc[s][i] = 0.f;
}

// Writes Y rows of the wave's queries: y[cc][i] = Y[query 4 g + i][column 16 cc + l % 16].
__device__ __forceinline__ void store_y(const FwdParams& p, const BlockCtx& c, const f32x4_t y[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = c.qt * kTile + c.wave * 16 + 4 * c.g + i;
    if (row < c.n) {
      float* yrow = p.Y + ((int64_t)c.b * c.n + row) * c.d_out + c.h * kDHead + c.r16;
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) yrow[16 * cc] = y[cc][i];
    }
  }
}

// ------------------------------------------------------------------ score pass
// The score pass computes S = Q K^T (Q as the MFMA A operand): lane (g, r16) of a wave
// holds the scores of its queries qw + 4 g + i (i < 4, qw = the wave's first query) with
// keys 16 s + r16 of each tile, so the statistics of a query row reduce over the 16 lanes
// of a lane row and the column max of a key reduces over four values in registers and the
// four lane rows. Softmax statistics are kept per query as c = M + log2(sum of exp2(logit -
// M)), so that A = exp2(dot a log2(e) - c) (one fma, one exp2; the output pass computes A
// the same way), and the column max is taken on t = dot a log2(e) - c before a single exp2
// per key: m = exp2(max t) = max A, because exp2 is monotone.

// The wave's four queries of lane row g under a local window: each attends keys
// klo .. klo + kspan (its window cut to the valid keys; all of them for query 0) and key 0.
struct RowQ {
  int klo[4], kspan[4];
};

template <bool BAND>
__device__ __forceinline__ RowQ row_queries(const BlockCtx& c) {
  RowQ r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r.klo[i] = 0;
    r.kspan[i] = 0;
    if constexpr (BAND) {
      const int q = c.qt * kTile + c.wave * 16 + 4 * c.g + i;
      int lo = q == 0 ? 0 : max(0, q - c.half);
      int hi = q == 0 ? c.len - 1 : min(c.len - 1, q + c.half);
      if (hi < lo) lo = hi = 1 << 30;  // a padded query past the window's reach: key 0 only
      r.klo[i] = lo;
      r.kspan[i] = hi - lo;
    }
  }
  return r;
}

// Key 16 s + r16 of tile kt (lim = len - 64 kt) is attended by query i of the lane row.
template <bool BAND>
__device__ __forceinline__ bool key_ok_q(const BlockCtx& c, const RowQ& rq, int kt, int lim, int s, int i) {
  if constexpr (BAND) {
    const bool in = (unsigned)(kt * kTile + 16 * s + c.r16 - rq.klo[i]) <= (unsigned)rq.kspan[i];
    return s == 0 ? (in || (kt == 0 && c.r16 == 0)) : in;
  } else {
    return lim >= kTile || 16 * s + c.r16 < lim;
  }
}

// Masks the scores of a tile the lane's queries do not all attend (a partial last tile, a
// local window): called only for such tiles, so that full tiles pay no per-key test.
template <bool BAND>
__device__ __forceinline__ void mask_tile_q(f32x4_t acc[4], const BlockCtx& c, const RowQ& rq, int kt, int lim,
                                            float fill) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (!key_ok_q<BAND>(c, rq, kt, lim, s, i)) acc[s][i] = fill;
}

// Offset of the column-max argument of query i: c (full attention) or c - log2 |S_q|
// (local window, the count rule's per-row factor); +inf for padded queries (excluded).
template <bool BAND>
__device__ __forceinline__ float colmax_offset(const BlockCtx& c, const RowQ& rq, int i, float cq) {
  const int q = c.qt * kTile + c.wave * 16 + 4 * c.g + i;
  if (q >= c.len) return INFINITY;
  if constexpr (BAND) {
    const int nk = rq.kspan[i] + 1 + (rq.klo[i] > 0 ? 1 : 0);
    return cq - __builtin_amdgcn_logf((float)nk);
  } else {
    return cq;
  }
}

// S = Q K^T for the 64 keys in LDS: acc[s][i] = dot(query 4 g + i, key 16 s + r16).
__device__ __forceinline__ void score_tile_qk(f32x4_t acc[4], const uint16_t* Ks, const QFrag<1>& q, int r16,
                                              int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    acc[s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8_t b = *reinterpret_cast<const bf16x8_t*>(Ks + kv_at(16 * s + r16, 32 * ks + 8 * g));
      acc[s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q.v[ks], b, acc[s], 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void score_tile_qk(f32x4_t acc[4], const float* Ks, const QFrag<0>& q, int r16, int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    acc[s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const float* krow = Ks + (16 * s + r16) * kStrideF + 16 * g;
#pragma unroll
    for (int t = 0; t < 16; ++t)
      acc[s] = __builtin_amdgcn_mfma_f32_16x16x4f32(q.v[t], krow[t], acc[s], 0, 0, 0);
  }
}

// Reductions over the 16 lanes of a lane row (DPP butterflies; every lane gets the result).
template <int CTRL>
__device__ __forceinline__ float row_max_step(float v) { return vmax(v, dpp_f32<CTRL>(v)); }
__device__ __forceinline__ float row16_max_sel(float v) {
  return row_max_step<0x140>(row_max_step<0x141>(row_max_step<0x4E>(row_max_step<0xB1>(v))));
}
template <int CTRL>
__device__ __forceinline__ float row_sum_step(float v) { return v + dpp_f32<CTRL>(v); }
__device__ __forceinline__ float row16_sum(float v) {
  return row_sum_step<0x140>(row_sum_step<0x141>(row_sum_step<0x4E>(row_sum_step<0xB1>(v))));
}
// (reference, sum of exp2(logit - reference)) pairs of the 16 lanes of a row combined,
// rescaled to the larger reference; a lane with no attended key holds (-inf or a reference
// below every logit, 0).
template <int CTRL>
__device__ __forceinline__ void row_stat_step(float& M, float& L) {
  const float m2 = dpp_f32<CTRL>(M), l2 = dpp_f32<CTRL>(L);
  const float Mn = vmax(M, m2);
  const float a = M == -INFINITY ? 0.f : __fmul_rn(L, exp2_fast(__fsub_rn(M, Mn)));
  const float b = m2 == -INFINITY ? 0.f : __fmul_rn(l2, exp2_fast(__fsub_rn(m2, Mn)));
  L = a + b;
  M = Mn;
}

// Column statistic of one tile, t = dot a log2(e) - cc[i]: the max of t over the lane's four
// queries (max rule) or the sum of exp2(t) = A (mean rule), per key 16 s + r16, left in
// cml[g][r16][s] (the wave's slot of the tile) for the combination over the four lane rows
// and the four waves (col_combine).
template <int IMP>
__device__ __forceinline__ void tile_colstat(const f32x4_t acc[4], const float cc[4], float (*cml)[16][4],
                                             const BlockCtx& c) {
  float v[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if constexpr (IMP == 1) {
      float t = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) t += exp2_fast(__fmaf_rn(acc[s][i], kLog2eOver8, -cc[i]));
      v[s] = t;
    } else {
      float t[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) t[i] = __fmaf_rn(acc[s][i], kLog2eOver8, -cc[i]);
      v[s] = vmax(vmax3(t[0], t[1], t[2]), t[3]);
    }
  }
  *reinterpret_cast<float4*>(&cml[c.g][c.r16][0]) = make_float4(v[0], v[1], v[2], v[3]);
}

// The block's partial of key e (< 64) of a tile from its sixteen values (four waves x four
// lane rows) in a fixed order: exp2 of the max (max rule; SCALED: the values are dot - c / s
// and the max is multiplied by s first) or the sum (mean rule).
template <int IMP, bool SCALED = false>
__device__ __forceinline__ float col_combine(const float (*cmt)[4][16][4], int e) {
  const int r16 = e & 15, sk = e >> 4;
  float x[16];
#pragma unroll
  for (int w = 0; w < 4; ++w)
#pragma unroll
    for (int g = 0; g < 4; ++g) x[4 * w + g] = cmt[w][g][r16][sk];
  if constexpr (IMP == 1) {
    float a[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) a[w] = (x[4 * w] + x[4 * w + 1]) + (x[4 * w + 2] + x[4 * w + 3]);
    return (a[0] + a[1]) + (a[2] + a[3]);
  } else {
    const float a = vmax3(x[0], x[1], x[2]), b = vmax3(x[3], x[4], x[5]), d = vmax3(x[6], x[7], x[8]);
    const float f = vmax3(x[9], x[10], x[11]), g = vmax3(x[12], x[13], x[14]);
    const float m = vmax3(vmax3(a, b, d), vmax3(f, g, x[15]), a);
    return exp2_fast(SCALED ? __fmul_rn(m, kLog2eOver8) : m);
  }
}

// Four probabilities of queries q .. q + 3 (q a multiple of 4) of one key, at dst = the
// key's row + q: one 16-byte store when all four queries exist and the row is 16-byte
// aligned (n a multiple of 4), else one store per existing query.
__device__ __forceinline__ void store_probs4(float* dst, float a0, float a1, float a2, float a3, int q, int n) {
  if ((n & 3) == 0 && q + 3 < n) {
    *reinterpret_cast<float4*>(dst) = make_float4(a0, a1, a2, a3);
  } else {
    if (q < n) dst[0] = a0;
    if (q + 1 < n) dst[1] = a1;
    if (q + 2 < n) dst[2] = a2;
    if (q + 3 < n) dst[3] = a3;
  }
}

// Median rule: the probabilities of one tile, A = exp2(dot a log2(e) - c), into the per-key
// array acol[b n + key][h][query].
__device__ __forceinline__ void store_probs(const FwdParams& p, const BlockCtx& c, const f32x4_t acc[4], int kt,
                                            const float cq[4], int qw) {
  float* ac = p.acol + (int64_t)c.b * c.n * p.H * c.n;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int key = kt * kTile + 16 * s + c.r16;
    if (key < c.n) {
      float a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = exp2_fast(__fmaf_rn(acc[s][i], kLog2eOver8, -cq[i]));
      store_probs4(ac + ((int64_t)key * p.H + c.h) * c.n + qw, a[0], a[1], a[2], a[3], qw, c.n);
    }
  }
}

// c of query qw + 4 g + i from lane r16 = i of each lane row.
__device__ __forceinline__ void store_row_c(const FwdParams& p, const BlockCtx& c, const float cq[4]) {
  const int q = c.qt * kTile + c.wave * 16 + 4 * c.g + c.r16;
  if (c.r16 < 4 && q < c.n) {
    const float v = c.r16 == 0 ? cq[0] : c.r16 == 1 ? cq[1] : c.r16 == 2 ? cq[2] : cq[3];
    p.row_c[((int64_t)c.b * p.H + c.h) * c.n + q] = v;
  }
}

// Resident variant: all ntl <= NT tiles in LDS and all scores in registers.
template <int BF, int NT, bool BAND, int IMP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void k_scores_res(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int S = stride_of<BF>();
  __shared__ __align__(16) T Ks[NT][kTile * S];
  __shared__ __align__(16) float cm[NT][4][4][16][4];  // [tile][wave][lane row][r16][s]
  const BlockCtx c = block_ctx(p);
  const T* Qb = static_cast<const T*>(p.Q) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const T* Kb = static_cast<const T*>(p.K) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;

  TileRegs kr[NT];
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) kr[kt] = tile_load<BF>(Kb, c.d_out, min(kt, c.ntl - 1) * kTile, c.n, c.tid);
  QFrag<BF> qf;
  load_qfrag(qf, Qb + (int64_t)min(c.q, c.n - 1) * c.d_out, c.g);
#pragma unroll
  for (int kt = 0; kt < NT; ++kt)
    if (kt < c.ntl) tile_store<BF>(kr[kt], Ks[kt], c.tid);
  lds_barrier();

  // scores in registers (masked keys -inf), the lane's max dot product per query
  const RowQ rq = row_queries<BAND>(c);
  f32x4_t acc[NT][4];
  float dmax[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    if (kt < c.ntl) {
      score_tile_qk(acc[kt], Ks[kt], qf, c.r16, c.g);
      const int lim = c.len - kt * kTile;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i)  // a select per key: cheaper here than a branch per tile
          acc[kt][s][i] = key_ok_q<BAND>(c, rq, kt, lim, s, i) ? acc[kt][s][i] : -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        dmax[i] = vmax3(vmax3(dmax[i], acc[kt][0][i], acc[kt][1][i]), acc[kt][2][i], acc[kt][3][i]);
    }
  }
  // row statistics: M = the largest logit (rounding is monotone, so it is the rounded
  // largest dot product), then the sum of exp2(logit - M) over the row's 16 lanes
  float M[4], Ls[4], cq[4], cc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    M[i] = __fmul_rn(row16_max_sel(dmax[i]), kLog2eOver8);  // finite: key 0 is attended
    Ls[i] = 0.f;
  }
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    if (kt < c.ntl) {
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) Ls[i] += exp2_fast(__fmaf_rn(acc[kt][s][i], kLog2eOver8, -M[i]));
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    cq[i] = M[i] + __builtin_amdgcn_logf(row16_sum(Ls[i]));
    cc[i] = colmax_offset<BAND>(c, rq, i, cq[i]);
  }
  store_row_c(p, c, cq);

  // column max (or, mean rule, column sum) of the block's valid queries, every tile in its
  // own LDS slot (one barrier); median rule: every probability to acol as well
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    if (kt < c.ntl) {
      tile_colstat<IMP>(acc[kt], cc, cm[kt][c.wave], c);
      if constexpr (IMP == 2) store_probs(p, c, acc[kt], kt, cq, c.qt * kTile + c.wave * 16 + 4 * c.g);
    }
  }
  lds_barrier();
  float* part = p.colmax_part + (int64_t)c.b * c.n * p.nparts + c.h * p.qtiles + c.qt;
  for (int e = c.tid; e < c.ntl * kTile; e += kThreads) {
    const float v = col_combine<IMP>(cm[e / kTile], e % kTile);
    if (e < c.n) part[(int64_t)e * p.nparts] = v;
  }
}

// Streamed-resident variant (up to NT visited tiles, padded length <= 64 NT): K tiles are
// streamed through two LDS buffers as in the streaming variant, but every score stays in
// registers, so a single sweep over K gives the statistics and the column statistic (the
// streaming variant computes every score twice and keeps online statistics).
template <int BF, int NT, bool BAND, int IMP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_scores_rs(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int S = stride_of<BF>();
  __shared__ __align__(16) T Ks[2][kTile * S];
  __shared__ __align__(16) float cm[NT][4][4][16][4];  // [tile][wave][lane row][r16][s]
  const BlockCtx c = block_ctx(p);
  const T* Qb = static_cast<const T*>(p.Q) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const T* Kb = static_cast<const T*>(p.K) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const int nvis = tile_count(c);  // <= NT (the launch checks the padded length)
  // two K tiles in flight: the work per tile before its buffer's barrier is short
  TileRegs kr = tile_load<BF>(Kb, c.d_out, 0, c.n, c.tid);
  TileRegs kr2 = tile_load<BF>(Kb, c.d_out, tile_at(c, min(1, nvis - 1)) * kTile, c.n, c.tid);
  QFrag<BF> qf;
  load_qfrag(qf, Qb + (int64_t)min(c.q, c.n - 1) * c.d_out, c.g);
  const RowQ rq = row_queries<BAND>(c);

  // scores in registers (masked keys -inf); the t-th visited tile goes through K buffer
  // t & 1 (the barrier after its store also orders the reads of tile t - 2, consumed by
  // that tile's MFMAs, before it). The row sums are software pipelined: once the MFMAs of
  // tile t are issued, the terms of tile t - 1 are added, under a reference M that is the
  // row's largest logit in tile 0 (finite: key 0 is attended by every query). A sum of
  // positive terms keeps its relative precision when terms exceed 1; only a logit more than
  // about 127 log2 units above M overflows it, and then (or with non-finite scores) the
  // wave takes each row's largest logit as M and sums again (a wave-uniform branch).
  f32x4_t acc[NT][4];
  float M[4], Ls[4] = {0.f, 0.f, 0.f, 0.f};
  auto tile0_ref = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      M[i] = __fmul_rn(row16_max_sel(vmax(vmax3(acc[0][0][i], acc[0][1][i], acc[0][2][i]), acc[0][3][i])),
                       kLog2eOver8);
  };
  auto add_terms = [&](const f32x4_t a[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) Ls[i] += exp2_fast(__fmaf_rn(a[s][i], kLog2eOver8, -M[i]));
  };
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t < nvis) {
      const int kt = tile_at(c, t);
      T* buf = Ks[t & 1];
      tile_store<BF>(kr, buf, c.tid);
      lds_barrier();
      kr = kr2;
      kr2 = tile_load<BF>(Kb, c.d_out, tile_at(c, min(t + 2, nvis - 1)) * kTile, c.n, c.tid);
      score_tile_qk(acc[t], buf, qf, c.r16, c.g);
      const int lim = c.len - kt * kTile;
      if (BAND || lim < kTile) mask_tile_q<BAND>(acc[t], c, rq, kt, lim, -INFINITY);  // tile-uniform
      if (t > 0) {
        if (t == 1) tile0_ref();
        add_terms(acc[t - 1]);
      }
    }
  }
  if (nvis == 1) tile0_ref();
#pragma unroll
  for (int t = 0; t < NT; ++t)
    if (t == nvis - 1) add_terms(acc[t]);
  float Lr[4], cq[4], cc[4];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    Lr[i] = row16_sum(Ls[i]);
    bad |= !(Lr[i] < INFINITY);
  }
  if (__any(bad)) {
    float dmax[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t < nvis) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          dmax[i] = vmax3(vmax3(dmax[i], acc[t][0][i], acc[t][1][i]), acc[t][2][i], acc[t][3][i]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      M[i] = __fmul_rn(row16_max_sel(dmax[i]), kLog2eOver8);
      Ls[i] = 0.f;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if (t < nvis) add_terms(acc[t]);
#pragma unroll
    for (int i = 0; i < 4; ++i) Lr[i] = row16_sum(Ls[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    cq[i] = M[i] + __builtin_amdgcn_logf(Lr[i]);
    cc[i] = colmax_offset<BAND>(c, rq, i, cq[i]);
  }
  store_row_c(p, c, cq);

  float* part = p.colmax_part + (int64_t)c.b * c.n * p.nparts + c.h * p.qtiles + c.qt;
  if (BAND) {  // valid keys of the tiles outside the window get a zero partial
    for (int key = kTile + c.tid; key < c.len; key += kThreads) {
      const int kt = key / kTile;
      if (kt < c.tlo || kt > c.thi) part[(int64_t)key * p.nparts] = 0.f;
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t < nvis) {
      tile_colstat<IMP>(acc[t], cc, cm[t][c.wave], c);
      if constexpr (IMP == 2) store_probs(p, c, acc[t], tile_at(c, t), cq, c.qt * kTile + c.wave * 16 + 4 * c.g);
    }
  }
  lds_barrier();
  for (int e = c.tid; e < nvis * kTile; e += kThreads) {
    const int t = e / kTile, k = e % kTile;
    const float v = col_combine<IMP>(cm[t], k);
    const int key = tile_at(c, t) * kTile + k;
    if (key < c.n) part[(int64_t)key * p.nparts] = v;
  }
}

// ------------------------------------------------------------------ Y = A H~
template <int BF, int NT, bool BAND>
__global__ __launch_bounds__(kThreads) void k_attn_res(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int S = stride_of<BF>();
  __shared__ __align__(16) T Ks[NT][kTile * S];
  __shared__ __align__(16) T Vs[NT][kTile * S];  // [key][column]
  const BlockCtx c = block_ctx(p);
  const int64_t off = (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const T* Qb = static_cast<const T*>(p.Q) + off;
  const T* Kb = static_cast<const T*>(p.K) + off;
  const T* Vb = static_cast<const T*>(p.Henc) + off;

  TileRegs kr[NT], vr[NT];
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    kr[kt] = tile_load<BF>(Kb, c.d_out, min(kt, c.ntl - 1) * kTile, c.n, c.tid);
    vr[kt] = tile_load<BF>(Vb, c.d_out, min(kt, c.ntl - 1) * kTile, c.n, c.tid);
  }
  QFrag<BF> qf;
  load_qfrag(qf, Qb + (int64_t)min(c.q, c.n - 1) * c.d_out, c.g);
  const int64_t so = ((int64_t)c.b * p.H + c.h) * c.n + min(c.q, c.n - 1);
  const float cq = p.row_c[so];
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    if (kt < c.ntl) {
      tile_store<BF>(kr[kt], Ks[kt], c.tid);
      tile_store_v<BF>(vr[kt], Vs[kt], c.tid);
    }
  }
  lds_barrier();

  f32x4_t y[4];
#pragma unroll
  for (int cc = 0; cc < 4; ++cc) y[cc] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kt = 0; kt < NT; ++kt) {
    if (kt < c.ntl) {
      f32x4_t acc[4];
      score_tile(acc, Ks[kt], qf, c.r16, c.g);
      const int lim = c.len - kt * kTile;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[s][i] = exp2_fast(__fmaf_rn(acc[s][i], kLog2eOver8, -cq));
      if (BAND || lim < kTile) mask_tile<BAND>(acc, c, kt, lim);  // tile-uniform
      pv_tile(y, acc, Vs[kt], c.r16, c.g);
    }
  }
  store_y(p, c, y);
}

// ------------------------------------------------------------------ Y = A H~, streaming
// The streaming output pass takes MT 16-query tiles per wave (64 MT queries per block):
// each K and H~ fragment read from LDS feeds MT MFMAs. With one query tile per wave the
// pass is bound by LDS reads; two cut its time by about a sixth at 4096 keys; three or
// four measured slower (fewer waves fit beside their accumulators), so MT = 2.

// Block context for blocks of QB queries (QB / 4 per wave); as block_ctx otherwise.
template <int QB>
__device__ __forceinline__ BlockCtx block_ctx_q(const FwdParams& p) {
  BlockCtx c;
  const int bid = blockIdx.x, Q = (p.n + QB - 1) / QB, P = p.H * p.B;
  int pair;
  if (P % 8 == 0) {  // the query tiles of a (batch row, head) on one XCD, as in block_ctx
    const int G = 8 * Q, w = bid % G;
    pair = bid / G * 8 + w % 8;
    c.qt = w / 8;
  } else {
    pair = bid / Q;
    c.qt = bid % Q;
  }
  c.h = pair % p.H;
  c.b = pair / p.H;
  c.tid = threadIdx.x;
  c.wave = c.tid >> 6;
  c.lane = c.tid & 63;
  c.r16 = c.lane & 15;
  c.g = c.lane >> 4;
  c.n = p.n;
  c.d_out = p.d_out;
  c.len = valid_len(p, c.b);
  c.q = c.qt * QB + c.wave * (QB / 4) + c.r16;  // query tile 0 of the wave; tile m is q + 16 m
  c.ntl = (c.len + kTile - 1) / kTile;
  c.half = p.band_half;
  c.tlo = 1;
  c.thi = c.ntl - 1;
  c.klo = 0;
  c.kspan = 0;
  if (c.half > 0 && c.qt > 0) {  // the window of queries q0 .. q0 + QB - 1
    const int q0 = c.qt * QB;
    c.tlo = max(1, max(q0 - c.half, 0) / kTile);
    c.thi = min(c.ntl - 1, (q0 + QB - 1 + c.half) / kTile);
  }
  return c;
}

// The window of query q (klo .. klo + kspan, and key 0), as block_ctx sets it for c.q.
// Under a local window: whether every key of tile kt is attended by every query q0 .. q0 +
// nq - 1 (then the tile needs no mask): the keys are below len and within half of each of
// those queries (query 0 attends every key below len). Wave-uniform arguments.
__device__ __forceinline__ bool band_tile_inside(const BlockCtx& c, int kt, int q0, int nq) {
  const int k0 = kt * kTile, k1 = k0 + kTile - 1;
  return k1 < c.len && k0 >= q0 + nq - 1 - c.half && k1 <= max(q0, 1) + c.half;
}

__device__ __forceinline__ void query_window(const BlockCtx& c, int q, int& klo, int& kspan) {
  int lo = q == 0 ? 0 : max(0, q - c.half);
  int hi = q == 0 ? c.len - 1 : min(c.len - 1, q + c.half);
  if (hi < lo) lo = hi = 1 << 30;
  klo = lo;
  kspan = hi - lo;
}

// S^T = K Q^T for MT 16-query tiles sharing each K fragment read.
template <int MT>
__device__ __forceinline__ void score_tile_m(f32x4_t acc[MT][4], const uint16_t* Ks, const QFrag<1> q[MT], int r16,
                                             int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m][s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(Ks + kv_at(16 * s + r16, 32 * ks + 8 * g));
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, q[m].v[ks], acc[m][s], 0, 0, 0);
    }
  }
}

template <int MT>
__device__ __forceinline__ void score_tile_m(f32x4_t acc[MT][4], const float* Ks, const QFrag<0> q[MT], int r16,
                                             int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m][s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const float* krow = Ks + (16 * s + r16) * kStrideF + 16 * g;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const float a = krow[t];
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, q[m].v[t], acc[m][s], 0, 0, 0);
    }
  }
}

// P V for MT query tiles sharing each H~ fragment read.
template <int MT>
__device__ __forceinline__ void pv_tile_m(f32x4_t y[MT][4], const f32x4_t acc[MT][4], const uint16_t* Vs, int r16,
                                          int g) {
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    bf16x8_t a[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
      a[m] = __builtin_bit_cast(bf16x8_t, make_uint4(pack_bf16x2(acc[m][2 * pp][0], acc[m][2 * pp][1]),
                                                     pack_bf16x2(acc[m][2 * pp][2], acc[m][2 * pp][3]),
                                                     pack_bf16x2(acc[m][2 * pp + 1][0], acc[m][2 * pp + 1][1]),
                                                     pack_bf16x2(acc[m][2 * pp + 1][2], acc[m][2 * pp + 1][3])));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint16_t* vrow = Vs + (32 * pp + 4 * g + (r16 >> 2)) * kStrideBfWide + 16 * c + 4 * (r16 & 3);
      const uint2 lo = lds_read_tr16(vrow);
      const uint2 hi = lds_read_tr16(vrow + 16 * kStrideBfWide);
      const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
      for (int m = 0; m < MT; ++m) y[m][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[m], bv, y[m][c], 0, 0, 0);
    }
  }
}

template <int MT>
__device__ __forceinline__ void pv_tile_m(f32x4_t y[MT][4], const f32x4_t acc[MT][4], const float* Vs, int r16,
                                          int g) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* vrow = Vs + (16 * s + 4 * g + i) * kStrideF + r16;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float v = vrow[16 * c];
#pragma unroll
        for (int m = 0; m < MT; ++m) y[m][c] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[m][s][i], v, y[m][c], 0, 0, 0);
      }
    }
}

// Software pipelined like the streaming score pass: iteration t issues the Q K^T MFMAs of tile
// t + 1 before the VALU work (exp2, bf16 packing) on tile t's scores and tile t's P V MFMAs.
// K and H~ tiles are double buffered in LDS with different schedules: K tile t + 1 is
// stored before iteration t's barrier (its buffer was last read by the Q K^T of tile t - 1,
// issued in iteration t - 2), H~ tile t + 1 after it (its buffer was last read by the P V of
// tile t - 1 in iteration t - 1, which every wave has finished once it passes the barrier).
// The bf16 full-attention instance is held to 168 registers (three waves per SIMD), which it
// meets without spilling; the others need more.
template <int BF, bool BAND, int MT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu((BF && !BAND) ? 3 : 1))) void k_attn_stream(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int S = stride_of<BF>();
  constexpr int QB = 64 * MT;  // queries per block
  __shared__ __align__(16) T Ks[2][kTile * S];
  constexpr int SV = BF ? kStrideBfWide : kStrideF;  // H~ tiles: unpermuted rows
  __shared__ __align__(16) T Vs[2][kTile * SV];
  BlockCtx c = block_ctx_q<QB>(p);
  const int qw = __builtin_amdgcn_readfirstlane(c.qt * QB + c.wave * (QB / 4));  // the wave's first query
  const int64_t off = (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const T* Qb = static_cast<const T*>(p.Q) + off;
  const T* Kb = static_cast<const T*>(p.K) + off;
  const T* Vb = static_cast<const T*>(p.Henc) + off;

  QFrag<BF> qf[MT];
  float cq[MT];
  int klo[MT], kspan[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int q = c.q + 16 * m;
    load_qfrag(qf[m], Qb + (int64_t)min(q, c.n - 1) * c.d_out, c.g);
    cq[m] = p.row_c[((int64_t)c.b * p.H + c.h) * c.n + min(q, c.n - 1)];
    klo[m] = 0;
    kspan[m] = 0;
    if (BAND) query_window(c, q, klo[m], kspan[m]);
  }

  f32x4_t y[MT][4];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) y[m][cc] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nvis = tile_count(c);
  TileRegs kr = tile_load<BF>(Kb, c.d_out, 0, c.n, c.tid);
  TileRegs vr = tile_load<BF>(Vb, c.d_out, 0, c.n, c.tid);
  tile_store<BF>(kr, Ks[0], c.tid);
  tile_store_v<BF, true>(vr, Vs[0], c.tid);
  const int t1 = tile_at(c, min(1, nvis - 1)) * kTile;
  kr = tile_load<BF>(Kb, c.d_out, t1, c.n, c.tid);
  vr = tile_load<BF>(Vb, c.d_out, t1, c.n, c.tid);
  lds_barrier();
  f32x4_t accA[MT][4], accB[MT][4];
  score_tile_m<MT>(accA, Ks[0], qf, c.r16, c.g);
  auto step = [&](f32x4_t cur[MT][4], f32x4_t nxt[MT][4], int t) {
    const int kt = tile_at(c, t);
    const int lim = c.len - kt * kTile;
    // tile-uniform: masked scores give probability 0; under a window, tiles that every query
    // of the wave attends whole need no mask
    if (__builtin_expect(BAND ? !band_tile_inside(c, kt, qw, QB / 4) : lim < kTile, 0)) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        c.klo = klo[m];
        c.kspan = kspan[m];
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (!key_ok<BAND>(c, kt, lim, s, i)) cur[m][s][i] = -INFINITY;
      }
    }
    const int nb = (t + 1) & 1;
    tile_store<BF>(kr, Ks[nb], c.tid);
    lds_barrier();
    tile_store_v<BF, true>(vr, Vs[nb], c.tid);
    const int next = tile_at(c, min(t + 2, nvis - 1)) * kTile;
    kr = tile_load<BF>(Kb, c.d_out, next, c.n, c.tid);
    vr = tile_load<BF>(Vb, c.d_out, next, c.n, c.tid);
    score_tile_m<MT>(nxt, Ks[nb], qf, c.r16, c.g);  // tile t + 1 (the last iteration repeats a tile, unused)
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) cur[m][s][i] = exp2_fast(__fmaf_rn(cur[m][s][i], kLog2eOver8, -cq[m]));
    pv_tile_m<MT>(y, cur, Vs[t & 1], c.r16, c.g);
  };
  int t = 0;
  for (; t + 1 < nvis; t += 2) {
    step(accA, accB, t);
    step(accB, accA, t + 1);
  }
  if (t < nvis) step(accA, accB, t);
  // y[m][cc][i] = Y[query c.q - r16 + 16 m + 4 g + i][column 16 cc + r16]
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = c.qt * QB + c.wave * (QB / 4) + 16 * m + 4 * c.g + i;
      if (row < c.n) {
        float* yrow = p.Y + ((int64_t)c.b * c.n + row) * c.d_out + c.h * kDHead + c.r16;
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) yrow[16 * cc] = y[m][cc][i];
      }
    }
}

// ------------------------------------------------------------------ score pass, streaming
// Streaming score pass (rows longer than 8 key tiles): 128 queries per block, two 16-query
// tiles per wave, so that every K fragment read from LDS feeds two MFMAs and the per-tile
// work (tile loads and stores, barriers, lane swaps, partial stores) serves twice the
// queries. Two sweeps over the visited tiles: per-lane row statistics, then the column
// statistic, one partial per (key, head, 128-query tile).
//
// Both sweeps are software pipelined: the MFMAs of tile t + 1 are issued before the VALU
// work on tile t's scores, so the matrix cores and the vector units of a wave work at the
// same time (a wave's MFMA results are only read one iteration later). The loop is unrolled
// by two so that the two accumulator sets swap roles without register copies.
//
// Sweep 2 folds the row normaliser into the MFMA: its accumulators start at -c_q / s
// (s = log2(e) / 8) instead of 0, so an accumulator holds dot - c_q / s, whose maximum over
// the lane's queries needs no per-score arithmetic; the maximum over the block is scaled by
// s once per key: t = s * max(dot - c_q / s) = max(dot s - c_q) (s > 0).

// S = Q K^T of two 16-query tiles: acc[m][s][i] = dot(query 16 m + 4 g + i, key 16 s + r16)
// + init[m][i].
__device__ __forceinline__ void score_tile_qk2(f32x4_t acc[2][4], const uint16_t* Ks, const QFrag<1> q[2], int r16,
                                               int g, const f32x4_t init[2]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const bf16x8_t b0 = *reinterpret_cast<const bf16x8_t*>(Ks + kv_at(16 * s + r16, 8 * g));
    const bf16x8_t b1 = *reinterpret_cast<const bf16x8_t*>(Ks + kv_at(16 * s + r16, 32 + 8 * g));
    acc[0][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q[0].v[0], b0, init[0], 0, 0, 0);
    acc[1][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q[1].v[0], b0, init[1], 0, 0, 0);
    acc[0][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q[0].v[1], b1, acc[0][s], 0, 0, 0);
    acc[1][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q[1].v[1], b1, acc[1][s], 0, 0, 0);
  }
}

__device__ __forceinline__ void score_tile_qk2(f32x4_t acc[2][4], const float* Ks, const QFrag<0> q[2], int r16,
                                               int g, const f32x4_t init[2]) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    acc[0][s] = init[0];
    acc[1][s] = init[1];
    const float* krow = Ks + (16 * s + r16) * kStrideF + 16 * g;
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const float b = krow[t];
      acc[0][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[0].v[t], b, acc[0][s], 0, 0, 0);
      acc[1][s] = __builtin_amdgcn_mfma_f32_16x16x4f32(q[1].v[t], b, acc[1][s], 0, 0, 0);
    }
  }
}

// IMP: the column statistic, 0 max (Eq. 8-9), 1 mean, 2 median (every probability to acol).
template <int BF, bool BAND, int IMP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_scores_stream(FwdParams p) {
  using T = typename Elem<BF>::T;
  constexpr int S = stride_of<BF>();
  __shared__ __align__(16) T Ks[2][kTile * S];
  // sweep 2: per tile (three in flight), per wave and lane row, the lane row's value of key
  // 16 s + r16 at [r16][s]
  __shared__ __align__(16) float cm[3][4][4][16][4];
  const BlockCtx c = block_ctx_q<128>(p);
  const T* Qb = static_cast<const T*>(p.Q) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const T* Kb = static_cast<const T*>(p.K) + (int64_t)c.b * c.n * c.d_out + c.h * kDHead;
  const int qw = __builtin_amdgcn_readfirstlane(c.qt * 128 + c.wave * 32);  // the wave's first query
  QFrag<BF> qf[2];
#pragma unroll
  for (int m = 0; m < 2; ++m) load_qfrag(qf[m], Qb + (int64_t)min(qw + 16 * m + c.r16, c.n - 1) * c.d_out, c.g);
  // the lane's eight queries qw + 16 m + 4 g + i in slot 4 m + i; under a local window each
  // attends keys klo .. klo + kspan and key 0
  int klo[8], kspan[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    klo[k] = 0;
    kspan[k] = 0;
    if constexpr (BAND) query_window(c, qw + 16 * (k >> 2) + 4 * c.g + (k & 3), klo[k], kspan[k]);
  }
  // masked keys of a tile the lane's queries do not all attend (called for such tiles only)
  auto mask = [&](f32x4_t acc[2][4], int kt, int lim) {
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bool ok;
          if constexpr (BAND) {
            const int key = kt * kTile + 16 * s + c.r16;
            ok = (unsigned)(key - klo[4 * m + i]) <= (unsigned)kspan[4 * m + i] || key == 0;
          } else {
            ok = 16 * s + c.r16 < lim;
          }
          if (!ok) acc[m][s][i] = -INFINITY;
        }
  };
  const int nvis = tile_count(c);
  // One sweep over the visited tiles, software pipelined: K tile t + 1 is staged in LDS buffer
  // (t + 1) & 1 and its scores issued on the matrix cores before `work` runs on tile t's
  // scores. The barrier of iteration t orders the LDS stores of tile t + 1 before their reads
  // and the reads of tile t - 1 (same buffer, two iterations earlier) before those stores.
  // Every iteration does the same (the last one stages and multiplies the last tile again,
  // with results unused): one straight-line region per tile, and a barrier in every iteration
  // (sweep 2 combines the waves' values of tile t - 1 after iteration t's barrier).
  // `first` sees tile 0's scores (masked) before the loop.
  auto sweep = [&](const f32x4_t init[2], auto&& first, auto&& work) {
    TileRegs kr = tile_load<BF>(Kb, c.d_out, 0, c.n, c.tid);
    tile_store<BF>(kr, Ks[0], c.tid);
    kr = tile_load<BF>(Kb, c.d_out, tile_at(c, min(1, nvis - 1)) * kTile, c.n, c.tid);
    lds_barrier();
    f32x4_t accA[2][4], accB[2][4];
    score_tile_qk2(accA, Ks[0], qf, c.r16, c.g, init);
    first(accA);
    auto step = [&](f32x4_t cur[2][4], f32x4_t nxt[2][4], int t) {
      const int kt = tile_at(c, t);
      const int lim = c.len - kt * kTile;
      if (BAND ? !band_tile_inside(c, kt, qw, 32) : lim < kTile) mask(cur, kt, lim);  // tile-uniform
      T* buf = Ks[(t + 1) & 1];
      tile_store<BF>(kr, buf, c.tid);
      lds_barrier();
      kr = tile_load<BF>(Kb, c.d_out, tile_at(c, min(t + 2, nvis - 1)) * kTile, c.n, c.tid);
      score_tile_qk2(nxt, buf, qf, c.r16, c.g, init);
      work(cur, t, kt);
    };
    int t = 0;
    for (; t + 1 < nvis; t += 2) {
      step(accA, accB, t);
      step(accB, accA, t + 1);
    }
    if (t < nvis) step(accA, accB, t);
  };

  // Sweep 1: per lane and query, a reference logit M and the sum of exp2(logit - M) over
  // the lane's keys; the 16 lanes of a row are combined at the end. M is the row's largest
  // logit in tile 0 (finite: key 0 is attended by every query), and every later term is
  // added under it, with no check per tile: the terms of a positive sum may exceed 1 without
  // losing relative precision, and only a logit more than 127 log2 units above M would
  // overflow. If any sum came out non-finite (that, or non-finite scores), the wave runs the
  // sweep again the careful way: terms added under the current reference as long as a tile's
  // four terms of a query sum to at most 2^16, otherwise (the first tile, and rarely later)
  // the tile redone with M raised to the running max and the sum rescaled. Both branches
  // are wave-uniform.
  constexpr float kNoMax = -1e30f;  // below every logit: no attended key seen yet
  constexpr float kRaise = 65536.f;
  float M[8], Ls[8];
  const f32x4_t zero2[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int k = 0; k < 8; ++k) Ls[k] = 0.f;
  sweep(
      zero2,
      [&](f32x4_t acc[2][4]) {
        if (BAND ? !band_tile_inside(c, 0, qw, 32) : c.len < kTile) mask(acc, 0, c.len);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int m = k >> 2, i = k & 3;
          const float dm = vmax(vmax3(acc[m][0][i], acc[m][1][i], acc[m][2][i]), acc[m][3][i]);
          M[k] = __fmul_rn(row16_max(dm), kLog2eOver8);
        }
      },
      [&](f32x4_t acc[2][4], int, int) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int m = k >> 2, i = k & 3;
          float e = exp2_fast(__fmaf_rn(acc[m][0][i], kLog2eOver8, -M[k]));
#pragma unroll
          for (int s = 1; s < 4; ++s) e += exp2_fast(__fmaf_rn(acc[m][s][i], kLog2eOver8, -M[k]));
          Ls[k] += e;
        }
      });
  bool overflow = false;
#pragma unroll
  for (int k = 0; k < 8; ++k) overflow |= !(Ls[k] < INFINITY);
  if (__any(overflow)) {
    lds_barrier();  // the first sweep is done with both K buffers
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      M[k] = kNoMax;
      Ls[k] = 0.f;
    }
    sweep(
        zero2, [&](f32x4_t[2][4]) {},
        [&](f32x4_t acc[2][4], int, int) {
          float ts[8];
          bool raise = false;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const int m = k >> 2, i = k & 3;
            float e = exp2_fast(__fmaf_rn(acc[m][0][i], kLog2eOver8, -M[k]));
#pragma unroll
            for (int s = 1; s < 4; ++s) e += exp2_fast(__fmaf_rn(acc[m][s][i], kLog2eOver8, -M[k]));
            ts[k] = e;
            raise |= !(e <= kRaise);
          }
          if (__any(raise)) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
              const int m = k >> 2, i = k & 3;
              const float dm = vmax(vmax3(acc[m][0][i], acc[m][1][i], acc[m][2][i]), acc[m][3][i]);
              const float Mn = vmax(M[k], __fmul_rn(dm, kLog2eOver8));
              float e = exp2_fast(__fmaf_rn(acc[m][0][i], kLog2eOver8, -Mn));
#pragma unroll
              for (int s = 1; s < 4; ++s) e += exp2_fast(__fmaf_rn(acc[m][s][i], kLog2eOver8, -Mn));
              Ls[k] = __fmul_rn(Ls[k], exp2_fast(__fsub_rn(M[k], Mn))) + e;
              M[k] = Mn;
            }
          } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) Ls[k] += ts[k];
          }
        });
  }
  float cq[8], cc[8];
  f32x4_t dneg[2];  // sweep 2's accumulator start: -cc / s per query (-inf for padded queries)
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    float Mi = M[k], Li = Ls[k];
    row_stat_step<0xB1>(Mi, Li);
    row_stat_step<0x4E>(Mi, Li);
    row_stat_step<0x141>(Mi, Li);
    row_stat_step<0x140>(Mi, Li);
    cq[k] = Mi + __builtin_amdgcn_logf(Li);  // finite: key 0 is attended by every query
    // the column statistic's offset: c, or c - log2 |S_q| under a window; +inf for
    // padded queries (excluded)
    const int q = qw + 16 * (k >> 2) + 4 * c.g + (k & 3);
    float off = cq[k];
    if constexpr (BAND) off = cq[k] - __builtin_amdgcn_logf((float)(kspan[k] + 1 + (klo[k] > 0 ? 1 : 0)));
    cc[k] = q >= c.len ? INFINITY : off;
    dneg[k >> 2][k & 3] = -__fdiv_rn(cc[k], kLog2eOver8);
  }
  {  // c of query qw + 16 m + 4 g + i from lane r16 = 4 m + i of each lane row
    float v = cq[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) v = c.r16 == k ? cq[k] : v;
    const int q = qw + 16 * (c.r16 >> 2) + 4 * c.g + (c.r16 & 3);
    if (c.r16 < 8 && q < c.n) p.row_c[((int64_t)c.b * p.H + c.h) * c.n + q] = v;
  }

  // Sweep 2: the per-key column statistic of this block's valid queries. Each lane row of each
  // wave leaves its value of tile t's keys (over its four queries of each of the wave's two
  // query tiles) in cm[t % 3][wave][row]; after the barrier of iteration t + 1 (or the final
  // one), threads 0..63 combine the sixteen values of a key in a fixed order and store the
  // block's partial. A slot is reused three tiles later, after two more barriers.
  float* part = p.colmax_part + (int64_t)c.b * c.n * p.nparts + c.h * p.qtiles + c.qt;
  if (BAND) {  // valid keys of the tiles outside the window get a zero partial
    for (int key = kTile + c.tid; key < c.len; key += kThreads) {
      const int kt = key / kTile;
      if (kt < c.tlo || kt > c.thi) part[(int64_t)key * p.nparts] = 0.f;
    }
  }
  constexpr bool sum = IMP == 1;
  auto combine = [&](int t) {  // the block's partial of tile t's keys
    if (c.tid < kTile) {
      const float r = col_combine<IMP == 1 ? 1 : 0, true>(cm[t % 3], c.tid);
      const int key = tile_at(c, t) * kTile + c.tid;
      if (key < c.n) part[(int64_t)key * p.nparts] = r;
    }
  };
  lds_barrier();  // sweep 1 is done with both K buffers
  sweep(dneg, [&](f32x4_t[2][4]) {}, [&](f32x4_t acc[2][4], int t, int kt) {
    // the lane's eight queries per key: the max of dot - cc / s (or the sum of the
    // probabilities exp2(s (dot - cc / s))), left in cm for the combination over the lane
    // rows and waves
    float v[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if constexpr (sum) {
        float e = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) e += exp2_fast(__fmul_rn(acc[k >> 2][s][k & 3], kLog2eOver8));
        v[s] = e;
      } else {
        v[s] = vmax3(vmax3(acc[0][s][0], acc[0][s][1], acc[0][s][2]), vmax3(acc[0][s][3], acc[1][s][0], acc[1][s][1]),
                     vmax(acc[1][s][2], acc[1][s][3]));
      }
    }
    *reinterpret_cast<float4*>(&cm[t % 3][c.wave][c.g][c.r16][0]) = make_float4(v[0], v[1], v[2], v[3]);
    if constexpr (IMP == 2) {  // median rule: every probability, exp2(s (dot - cc / s))
      float* ac = p.acol + (int64_t)c.b * c.n * p.H * c.n;
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int key = kt * kTile + 16 * s + c.r16;
          if (key < c.n) {
            const int q = qw + 16 * m + 4 * c.g;
            float a[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = exp2_fast(__fmul_rn(acc[m][s][i], kLog2eOver8));
            store_probs4(ac + ((int64_t)key * p.H + c.h) * c.n + q, a[0], a[1], a[2], a[3], q, c.n);
          }
        }
    }
    if (t > 0) combine(t - 1);  // the barrier of this iteration follows every wave's tile t - 1 values
  });
  lds_barrier();
  combine(nvis - 1);
}

template <int BF, bool BAND>
hipError_t launch_scores_stream(const FwdParams& p, hipStream_t s) {
  const dim3 grid((unsigned)(p.qtiles * p.H * p.B)), blk(kThreads);
  if constexpr (BAND) {  // the mean and median rules are defined for full attention only
    return launch_stage_kernel((k_scores_stream<BF, true, 0>), grid, blk, 0, s, p);
  } else {
    if (p.importance == 1) return launch_stage_kernel((k_scores_stream<BF, false, 1>), grid, blk, 0, s, p);
    if (p.importance == 2) return launch_stage_kernel((k_scores_stream<BF, false, 2>), grid, blk, 0, s, p);
    return launch_stage_kernel((k_scores_stream<BF, false, 0>), grid, blk, 0, s, p);
  }
}

// The one-sweep score passes with the importance rule as a template parameter (the mean and
// median rules are defined for full attention only).
template <int BF, int NT, bool BAND, bool RS>
hipError_t launch_scores_onesweep(const FwdParams& p, hipStream_t s) {
  const dim3 grid((unsigned)(p.qtiles * p.H * p.B)), blk(kThreads);
  if (!BAND && p.importance == 1) {
    if constexpr (RS) return launch_stage_kernel(k_scores_rs<BF, NT, BAND, 1>, grid, blk, 0, s, p);
    else return launch_stage_kernel(k_scores_res<BF, NT, BAND, 1>, grid, blk, 0, s, p);
  }
  if (!BAND && p.importance == 2) {
    if constexpr (RS) return launch_stage_kernel(k_scores_rs<BF, NT, BAND, 2>, grid, blk, 0, s, p);
    else return launch_stage_kernel(k_scores_res<BF, NT, BAND, 2>, grid, blk, 0, s, p);
  }
  if constexpr (RS) return launch_stage_kernel(k_scores_rs<BF, NT, BAND, 0>, grid, blk, 0, s, p);
  else return launch_stage_kernel(k_scores_res<BF, NT, BAND, 0>, grid, blk, 0, s, p);
}

// Resident variants for padded lengths up to 256 keys (bf16) or 128 keys (fp32), the
// one-sweep streamed variant up to 8 key tiles, the two-sweep streaming variant beyond.
template <bool BAND>
hipError_t launch_scores_band(const FwdParams& p, hipStream_t s) {
  const int nt = (p.n + kTile - 1) / kTile;
  if (p.bf16) {
    if (nt <= 1) return launch_scores_onesweep<1, 1, BAND, false>(p, s);
    else if (nt <= 2) return launch_scores_onesweep<1, 2, BAND, false>(p, s);
    else if (nt <= 4) return launch_scores_onesweep<1, 4, BAND, false>(p, s);
    else if (nt <= 8) return launch_scores_onesweep<1, 8, BAND, true>(p, s);
    else return launch_scores_stream<1, BAND>(p, s);
  } else {
    if (nt <= 1) return launch_scores_onesweep<0, 1, BAND, false>(p, s);
    else if (nt <= 2) return launch_scores_onesweep<0, 2, BAND, false>(p, s);
    else if (nt <= 8) return launch_scores_onesweep<0, 8, BAND, true>(p, s);
    else return launch_scores_stream<0, BAND>(p, s);
  }
}

template <bool BAND>
hipError_t launch_attn_band(const FwdParams& p, hipStream_t s) {
  const dim3 grid((unsigned)(p.qtiles * p.H * p.B)), blk(kThreads);
  const int nt = (p.n + kTile - 1) / kTile;
  if (p.bf16) {
    if (nt <= 1) return launch_stage_kernel((k_attn_res<1, 1, BAND>), grid, blk, 0, s, p);
    else if (nt <= 2) return launch_stage_kernel((k_attn_res<1, 2, BAND>), grid, blk, 0, s, p);
    else if (nt <= 4) return launch_stage_kernel((k_attn_res<1, 4, BAND>), grid, blk, 0, s, p);
    else return launch_stage_kernel((k_attn_stream<1, BAND, 2>), dim3((unsigned)(((p.n + 127) / 128) * p.H * p.B)),
                                    blk, 0, s, p);
  } else {
    if (nt <= 1) return launch_stage_kernel((k_attn_res<0, 1, BAND>), grid, blk, 0, s, p);
    else if (nt <= 2) return launch_stage_kernel((k_attn_res<0, 2, BAND>), grid, blk, 0, s, p);
    else return launch_stage_kernel((k_attn_stream<0, BAND, 2>), dim3((unsigned)(((p.n + 127) / 128) * p.H * p.B)),
                                    blk, 0, s, p);
  }
}
}  // namespace

hipError_t launch_scores_colmax(const FwdParams& p, hipStream_t s) {
  return p.band_half > 0 ? launch_scores_band<true>(p, s) : launch_scores_band<false>(p, s);
}

hipError_t launch_attn_out(const FwdParams& p, hipStream_t s) {
  return p.band_half > 0 ? launch_attn_band<true>(p, s) : launch_attn_band<false>(p, s);
}

}  // namespace mca
