// Device-side helpers shared by the MCA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mca {

constexpr int kDHead = 64;
constexpr int kWave = 64;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// ---------------------------------------------------------------- bf16 <-> f32
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// float32 -> bfloat16 with v_cvt_pk_bf16_f32: round to nearest, ties to even; NaN stays
// NaN (checked bit for bit against the integer rounding u + 0x7fff + ((u >> 16) & 1)).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}

// Load element i of a row of T as float (T = float or uint16_t holding bf16 bits).
__device__ __forceinline__ float load_f32(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_f32(const uint16_t* p, int64_t i) {
  return bf16_bits_to_f32(p[i]);
}

// Four consecutive elements (4-element aligned) as floats.
__device__ __forceinline__ float4 load4_f32(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4_f32(const uint16_t* p) {
  uint2 v = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                     __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}

// ---------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11).
// Round: (c0,c1,c2,c3) -> (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0));
// the key advances by the Weyl constants between rounds.
struct u32x4 { uint32_t x, y, z, w; };

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = (uint64_t)M0 * c.x;  // one v_mad_u64_u32 each: both halves
    const uint64_t p1 = (uint64_t)M1 * c.z;
    c = u32x4{(uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0};
    k0 += W0;
    k1 += W1;
  }
  return c;
}

// ---------------------------------------------------------------- block barrier
// Barrier for threads that communicate through LDS only: the fences are restricted to the
// LDS address space, so outstanding global loads (prefetches) stay in flight across it
// (__syncthreads would wait for them).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ---------------------------------------------------------------- DPP reductions
// Data-parallel-primitive lane moves within rows of 16 lanes (register-only, no LDS).
// Controls: quad_perm [1,0,3,2] = 0xB1, quad_perm [2,3,0,1] = 0x4E, row_half_mirror =
// 0x141, row_mirror = 0x140; each is a permutation of the row, so every lane has a source.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Max over the 16 lanes of a row (lanes 16k .. 16k+15); every lane of the row gets it.
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  return fmaxf(v, dpp_f32<0x140>(v));
}

// ---------------------------------------------------------------- wave reductions
// Inclusive prefix sums over the 64 lanes with DPP (no LDS): shifts by 1, 2, 4, 8 within
// rows of 16 lanes, then lane 15 of rows 0 and 2 into rows 1 and 3, then lane 31 into
// rows 2 and 3. Lanes without a source, and rows left out, add 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_or_zero(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t scan_step(uint32_t v) { return v + dpp_or_zero<CTRL, ROWS>(v); }
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t scan_step(uint64_t v) {
  const uint32_t lo = dpp_or_zero<CTRL, ROWS>((uint32_t)v), hi = dpp_or_zero<CTRL, ROWS>((uint32_t)(v >> 32));
  return v + (((uint64_t)hi << 32) | lo);
}
template <typename U>
__device__ __forceinline__ U wave_inclusive_scan(U v) {
  v = scan_step<0x111, 0xF>(v);  // row_shr:1
  v = scan_step<0x112, 0xF>(v);  // row_shr:2
  v = scan_step<0x114, 0xF>(v);  // row_shr:4
  v = scan_step<0x118, 0xF>(v);  // row_shr:8
  v = scan_step<0x142, 0xA>(v);  // row_bcast:15 into rows 1, 3
  v = scan_step<0x143, 0xC>(v);  // row_bcast:31 into rows 2, 3
  return v;
}

// Max over the 64 lanes (DPP within rows of 16, then the four row results), wave-uniform.
__device__ __forceinline__ float wave_max(float v) {
  v = row16_max(v);
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

}  // namespace mca
