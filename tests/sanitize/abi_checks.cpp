// Host-side checks of the C ABI (argument validation, sizes, status strings, profiler
// bookkeeping) for a build with AddressSanitizer and UndefinedBehaviorSanitizer on the host
// code. Every call here returns before any device work, so it runs without a GPU. Exit status
// 0 when every check holds; the sanitizers abort on the first report.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>

#include "mca.h"

static int failures = 0;
#define CHECK(cond)                                                     \
  do {                                                                  \
    if (!(cond)) {                                                      \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                       \
    }                                                                   \
  } while (0)

static mca_forward_desc base_desc() {
  mca_forward_desc d;
  std::memset(&d, 0, sizeof d);
  d.batch = 2;
  d.seq = 128;
  d.heads = 12;
  d.d_head = 64;
  d.d_in = 768;
  d.dtype = MCA_BF16;
  d.sampling = MCA_SAMPLING_TOKEN;
  d.alpha = 0.4;
  d.seed = 0;
  return d;
}

static mca_status ws_status(const mca_forward_desc& d) {
  size_t bytes = 0;
  return mca_workspace_size(&d, &bytes);
}

int main() {
  // status strings and stage names, including out-of-range values
  CHECK(std::strcmp(mca_status_string(MCA_OK), "MCA_OK") == 0);
  CHECK(std::strcmp(mca_status_string(99), "MCA_ERR_UNKNOWN") == 0);
  CHECK(std::strcmp(mca_status_string(-1), "MCA_ERR_UNKNOWN") == 0);
  CHECK(mca_num_stages() == MCA_NUM_STAGES);
  for (int s = -2; s < MCA_NUM_STAGES + 2; ++s) CHECK(mca_stage_name(s) != nullptr);

  // sizes
  size_t bytes = 0;
  mca_forward_desc d = base_desc();
  CHECK(mca_workspace_size(&d, &bytes) == MCA_OK && bytes > 0);
  CHECK(mca_workspace_size(&d, nullptr) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_workspace_size(nullptr, &bytes) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepared_size(MCA_F32, 768, 768, &bytes) == MCA_OK && bytes > 0);
  CHECK(mca_prepared_size(5, 768, 768, &bytes) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepared_size(MCA_F32, 0, 768, &bytes) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepared_size(MCA_F32, 768, 768, nullptr) == MCA_ERR_INVALID_ARGUMENT);
  d.importance = MCA_IMPORTANCE_MEDIAN;  // the largest layout (every probability per key)
  d.batch = 1 << 12;
  d.seq = 1 << 12;
  CHECK(mca_workspace_size(&d, &bytes) == MCA_OK && bytes > (size_t(1) << 36));

  // descriptor validation: every field out of range
  struct Case {
    void (*edit)(mca_forward_desc&);
    mca_status want;
  };
  const Case cases[] = {
      {[](mca_forward_desc& x) { x.alpha = 0.0; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.alpha = -1.0; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.alpha = std::numeric_limits<double>::quiet_NaN(); }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.alpha = std::numeric_limits<double>::infinity(); }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.batch = 0; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.seq = -5; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.batch = int64_t(1) << 40; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.seq = int64_t(1) << 62; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.heads = int64_t(1) << 62; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.d_in = 2049; }, MCA_ERR_UNSUPPORTED},
      {[](mca_forward_desc& x) { x.d_in = 0; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.heads = 3; }, MCA_ERR_UNSUPPORTED},
      {[](mca_forward_desc& x) { x.heads = 36; }, MCA_ERR_UNSUPPORTED},
      {[](mca_forward_desc& x) { x.d_head = 128; }, MCA_ERR_UNSUPPORTED},
      {[](mca_forward_desc& x) { x.dtype = 7; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.sampling = -1; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.window = 3; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.window = int64_t(1) << 40; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.importance = 9; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.importance = MCA_IMPORTANCE_MEAN; x.window = 64; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.exact_from = -3; }, MCA_ERR_INVALID_ARGUMENT},
      {[](mca_forward_desc& x) { x.colmax_out = reinterpret_cast<float*>(0x10004); }, MCA_ERR_INVALID_ARGUMENT},
  };
  for (const Case& c : cases) {
    mca_forward_desc x = base_desc();
    c.edit(x);
    CHECK(ws_status(x) == c.want);
    CHECK(std::strlen(mca_last_error()) > 0);
  }

  // forward entry points: null, misaligned and too-small arguments are rejected before any
  // device work (the pointers below are never dereferenced)
  d = base_desc();
  d.batch = 1;
  d.seq = 16;
  d.heads = 4;
  d.d_in = 64;
  CHECK(mca_workspace_size(&d, &bytes) == MCA_OK);
  void* fake = reinterpret_cast<void*>(0x10000);
  float* fy = static_cast<float*>(fake);
  int32_t* fr = static_cast<int32_t*>(fake);
  CHECK(mca_attention_forward(&d, nullptr, fake, fake, fake, fake, fy, fr, fake, bytes, nullptr) ==
        MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_attention_forward(&d, fake, fake, fake, fake, fake, fy, fr, fake, bytes - 1, nullptr) ==
        MCA_ERR_WORKSPACE_TOO_SMALL);
  CHECK(mca_attention_forward(&d, reinterpret_cast<void*>(0x10004), fake, fake, fake, fake, fy, fr, fake, bytes,
                              nullptr) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_attention_forward(nullptr, fake, fake, fake, fake, fake, fy, fr, fake, bytes, nullptr) ==
        MCA_ERR_INVALID_ARGUMENT);
  mca_forward_desc big = base_desc();
  big.batch = 4;
  big.seq = 4096;
  CHECK(mca_attention_forward_noalloc(&big, fake, fake, fake, fake, fake, fy, fr, nullptr) ==
        MCA_ERR_WORKSPACE_TOO_SMALL);
  mca_forward_desc withprof = d;
  withprof.profiler = fake;
  CHECK(mca_attention_forward_noalloc(&withprof, fake, fake, fake, fake, fake, fy, fr, nullptr) ==
        MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_attention_forward_noalloc(nullptr, fake, fake, fake, fake, fake, fy, fr, nullptr) ==
        MCA_ERR_INVALID_ARGUMENT);

  // weight preparation
  CHECK(mca_prepare_weights(nullptr, MCA_F32, 8, 8, fake, size_t(1) << 30, nullptr) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepare_weights(fake, MCA_F32, 4097, 8, fake, size_t(1) << 30, nullptr) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepare_weights(fake, MCA_F32, 8, 8, reinterpret_cast<void*>(0x10002), size_t(1) << 30, nullptr) ==
        MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_prepared_size(MCA_F32, 8, 8, &bytes) == MCA_OK);
  CHECK(mca_prepare_weights(fake, MCA_F32, 8, 8, fake, bytes - 1, nullptr) == MCA_ERR_INVALID_ARGUMENT);

  // profiler bookkeeping without recorded launches
  void* prof = nullptr;
  CHECK(mca_profiler_create(nullptr) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_profiler_create(&prof) == MCA_OK && prof != nullptr);
  double ms[MCA_NUM_STAGES];
  int64_t launches[MCA_NUM_STAGES];
  CHECK(mca_profiler_collect(prof, ms, launches, MCA_NUM_STAGES) == MCA_OK);
  for (int s = 0; s < MCA_NUM_STAGES; ++s) CHECK(ms[s] == 0.0 && launches[s] == 0);
  CHECK(mca_profiler_collect(prof, ms, launches, MCA_NUM_STAGES + 1) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_profiler_collect(nullptr, ms, launches, 1) == MCA_ERR_INVALID_ARGUMENT);
  CHECK(mca_profiler_destroy(prof) == MCA_OK);
  CHECK(mca_profiler_destroy(nullptr) == MCA_OK);

  if (failures) std::fprintf(stderr, "%d check(s) failed\n", failures);
  else std::printf("all ABI checks passed under the host sanitizers\n");
  return failures ? 1 : 0;
}
