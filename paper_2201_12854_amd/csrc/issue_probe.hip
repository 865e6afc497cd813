// Issue-cost probes for gfx950: measurement support for the roofline reasoning about the
// attention kernels, built into a library of its own (libmca_probe.so) and not part of the
// attention path. Every wave runs `rounds` rounds of a fixed block of independent
// instructions and stamps the shader clock (s_memtime) and the constant 100 MHz clock
// (s_memrealtime) before and after them; the host turns the stamps into cycles per
// instruction per SIMD and, for the matrix cores, a chip-wide rate.
//
// Kinds (per wave and round):
//   0 fma   64 v_fma_f32 (eight independent chains of eight)
//   1 exp   64 v_exp_f32 (eight independent chains of eight)
//   2 mfma  16 v_mfma_f32_16x16x32_bf16 (eight independent accumulators, two each)
//   3 mix   the 64 fma and the 16 mfma of kinds 0 and 2 in one wave
//   4 split waves 0..3 of the workgroup run kind 0, waves 4..7 kind 2: with two waves per
//           SIMD (512 threads) each SIMD holds one wave of each
//   5 exp+mfma  the 64 exp of kind 1 and the 16 mfma of kind 2 in one wave
//   6 exp|mfma  waves 0..3 run kind 1, waves 4..7 kind 2 (as kind 4)
//   7 max3  64 v_max3_f32 per round (eight independent chains of eight)
//   8 exp+fma   the 64 exp of kind 1 and 64 fma (eight more chains) in one wave
// One workgroup per CU: its dynamic LDS (kPadLds bytes, untouched) leaves no room for a
// second. 256 w threads per workgroup put w waves on each of the CU's four SIMDs.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "mca_probe.h"

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 probe_bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float probe_f32x4_t;

constexpr int kFma = 0, kExp = 1, kMfma = 2, kMix = 3, kSplit = 4, kExpMix = 5, kExpSplit = 6, kMax3 = 7, kExpFma = 8;
constexpr int kPadLds = 96 * 1024;
constexpr int kInputs = 128;  // floats of the input buffer

template <int KIND>
__global__ __launch_bounds__(1024) void k_issue(const float* in, float* out, long long* stamps, int rounds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float x = in[lane], y = in[64 + lane];
  float a[8], b[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    a[k] = x + (float)k;
    b[k] = y + (float)k;
  }
  probe_f32x4_t acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = probe_f32x4_t{0.f, 0.f, 0.f, 0.f};
  const uint32_t xb = __float_as_uint(x), yb = __float_as_uint(y);
  const probe_bf16x8_t A = __builtin_bit_cast(probe_bf16x8_t, make_uint4(xb, yb, xb, yb));
  const probe_bf16x8_t B = __builtin_bit_cast(probe_bf16x8_t, make_uint4(yb, xb, yb, xb));
  const bool do_fma = KIND == kFma || KIND == kMix || (KIND == kSplit && wave < 4);
  const bool do_exp = KIND == kExp || KIND == kExpMix || KIND == kExpFma || (KIND == kExpSplit && wave < 4);
  const bool do_mfma = KIND == kMfma || KIND == kMix || KIND == kExpMix || ((KIND == kSplit || KIND == kExpSplit) && wave >= 4);

  const long long t0 = (long long)__builtin_amdgcn_s_memtime();
  const long long r0 = (long long)__builtin_amdgcn_s_memrealtime();
  for (int r = 0; r < rounds; ++r) {
    if (do_exp) {  // wave-uniform
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) a[k] = __builtin_amdgcn_exp2f(a[k]);
    }
    if (KIND == kExpFma) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) b[k] = fmaf(b[k], x, y);
    }
    if (KIND == kMax3) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) a[k] = __builtin_fmaxf(__builtin_fmaxf(a[k], x), y + (float)j);
    }
    if (do_fma) {  // wave-uniform
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) a[k] = fmaf(a[k], x, y);
    }
    if (do_mfma) {  // wave-uniform
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[k], 0, 0, 0);
    }
  }
  const long long t1 = (long long)__builtin_amdgcn_s_memtime();
  const long long r1 = (long long)__builtin_amdgcn_s_memrealtime();

  float s = 0.f;  // every result stays live
#pragma unroll
  for (int k = 0; k < 8; ++k) s += a[k] + b[k] + acc[k][0] + acc[k][1] + acc[k][2] + acc[k][3];
  out[(int64_t)blockIdx.x * blockDim.x + tid] = s;
  if (lane == 0) {
    long long* st = stamps + ((int64_t)blockIdx.x * (blockDim.x >> 6) + wave) * 4;
    st[0] = t0;
    st[1] = t1;
    st[2] = r0;
    st[3] = r1;
  }
}

template <int KIND>
hipError_t launch_kind(dim3 grid, dim3 block, const float* in, float* out, long long* stamps, int rounds) {
  hipError_t e = hipFuncSetAttribute((const void*)k_issue<KIND>, hipFuncAttributeMaxDynamicSharedMemorySize, kPadLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_issue<KIND>, grid, block, kPadLds, 0, in, out, stamps, rounds);
  return hipGetLastError();
}

}  // namespace

// Runs one probe on the current device (arguments and results as declared in mca_probe.h).
extern "C" int mca_issue_probe(int kind, int waves_per_simd, int rounds, long long* stamps, int max_waves,
                               int* nwaves) {
  if (kind < 0 || kind > 8 || rounds < 1 || rounds > (1 << 20) || !stamps || !nwaves) return -1;
  if (waves_per_simd != 1 && waves_per_simd != 2 && waves_per_simd != 4) return -1;
  if ((kind == kSplit || kind == kExpSplit) && waves_per_simd != 2) return -1;
  int dev = 0, ncu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return (int)e;
  const int threads = 256 * waves_per_simd, nw = ncu * 4 * waves_per_simd;
  *nwaves = nw;
  if (nw > max_waves) return -1;
  float host_in[kInputs];
  for (int i = 0; i < 64; ++i) {
    host_in[i] = 1.0f + 1e-6f * (float)i;  // fma chains a * x + y stay finite over any rounds
    host_in[64 + i] = -1e-7f * (float)(i + 1);
  }
  float *in = nullptr, *out = nullptr;
  long long* st = nullptr;
  e = hipMalloc((void**)&in, sizeof(host_in));
  if (e == hipSuccess) e = hipMalloc((void**)&out, sizeof(float) * (size_t)ncu * threads);
  if (e == hipSuccess) e = hipMalloc((void**)&st, sizeof(long long) * 4 * (size_t)nw);
  if (e == hipSuccess) e = hipMemcpy(in, host_in, sizeof(host_in), hipMemcpyHostToDevice);
  if (e == hipSuccess) {
    const dim3 grid((unsigned)ncu), block((unsigned)threads);
    switch (kind) {
      case kFma: e = launch_kind<kFma>(grid, block, in, out, st, rounds); break;
      case kExp: e = launch_kind<kExp>(grid, block, in, out, st, rounds); break;
      case kMfma: e = launch_kind<kMfma>(grid, block, in, out, st, rounds); break;
      case kMix: e = launch_kind<kMix>(grid, block, in, out, st, rounds); break;
      case kSplit: e = launch_kind<kSplit>(grid, block, in, out, st, rounds); break;
      case kExpMix: e = launch_kind<kExpMix>(grid, block, in, out, st, rounds); break;
      case kExpSplit: e = launch_kind<kExpSplit>(grid, block, in, out, st, rounds); break;
      case kMax3: e = launch_kind<kMax3>(grid, block, in, out, st, rounds); break;
      default: e = launch_kind<kExpFma>(grid, block, in, out, st, rounds); break;
    }
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipMemcpy(stamps, st, sizeof(long long) * 4 * (size_t)nw, hipMemcpyDeviceToHost);
  if (in) (void)hipFree(in);
  if (out) (void)hipFree(out);
  if (st) (void)hipFree(st);
  return e == hipSuccess ? 0 : (int)e;
}
