// C ABI of libmca: argument checks, workspace layout, stage launches, profiler.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "mca.h"
#include "mca_kernels.h"

namespace {

thread_local char g_last_error[512] = "";

mca_status fail(mca_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

mca_status ok() {
  g_last_error[0] = '\0';
  return MCA_OK;
}

constexpr int64_t kMaxDin = 2048;
constexpr int64_t kMaxDout = 2048;
constexpr int64_t kMaxTokens = int64_t(1) << 30;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

struct Layout {
  size_t colmax_part, row_c, henc, list, ucount, acol, total;
  int qtiles, nparts;
};

Layout layout_for(const mca_forward_desc& d) {
  const size_t tokens = size_t(d.batch) * size_t(d.seq);
  const size_t d_out = size_t(d.heads) * 64;
  const size_t helem = d.dtype == MCA_BF16 ? 2 : 4;
  Layout L;
  const int qt = mca::score_query_tile((int)d.seq);
  L.qtiles = (int)((d.seq + qt - 1) / qt);
  L.nparts = (int)(d.heads * L.qtiles);
  size_t off = 0;
  L.colmax_part = off; off = align256(off + 4 * tokens * size_t(L.nparts));
  L.row_c = off;       off = align256(off + 4 * tokens * size_t(d.heads));
  L.henc = off;        off = align256(off + helem * tokens * d_out);
  L.list = off;
  off = align256(off + 8 * (tokens * size_t(mca::list_stride((int)d.d_in)) + size_t(mca::list_tail_pad((int)d.d_in))));
  L.ucount = off;      off = align256(off + 4 * tokens);
  L.acol = off;        // median rule: every attention probability, per key
  if (d.importance == MCA_IMPORTANCE_MEDIAN) off = align256(off + 4 * tokens * size_t(d.heads) * size_t(d.seq));
  L.total = off;
  return L;
}

mca_status check_desc(const mca_forward_desc* d) {
  if (!d) return fail(MCA_ERR_INVALID_ARGUMENT, "desc is NULL");
  if (d->batch < 1 || d->seq < 1 || d->heads < 1 || d->d_in < 1 || d->d_head < 1)
    return fail(MCA_ERR_INVALID_ARGUMENT, "batch, seq, heads, d_head and d_in must be >= 1");
  if (d->sampling != MCA_SAMPLING_TOKEN && d->sampling != MCA_SAMPLING_WEIGHT)
    return fail(MCA_ERR_INVALID_ARGUMENT, "sampling %d is not MCA_SAMPLING_TOKEN or MCA_SAMPLING_WEIGHT", d->sampling);
  if (d->dtype != MCA_F32 && d->dtype != MCA_BF16)
    return fail(MCA_ERR_INVALID_ARGUMENT, "dtype %d is not MCA_F32 or MCA_BF16", d->dtype);
  if (d->window < 0 || d->window % 2 != 0 || d->window > (int64_t(1) << 25))
    return fail(MCA_ERR_INVALID_ARGUMENT, "window must be 0 or an even number of keys in 2..2^25 (got %lld)",
                (long long)d->window);
  if (d->importance < MCA_IMPORTANCE_MAX || d->importance > MCA_IMPORTANCE_MEDIAN)
    return fail(MCA_ERR_INVALID_ARGUMENT, "importance %d is not an mca_importance", d->importance);
  if (d->exact_from < 0) return fail(MCA_ERR_INVALID_ARGUMENT, "exact_from must be >= 0 (got %d)", d->exact_from);
  if (d->importance != MCA_IMPORTANCE_MAX && d->window != 0)
    return fail(MCA_ERR_INVALID_ARGUMENT, "the mean and median rules are defined for full attention (window 0)");
  if (!std::isfinite(d->alpha) || !(d->alpha > 0.0))
    return fail(MCA_ERR_INVALID_ARGUMENT, "alpha must be finite and > 0 (got %g)", d->alpha);
  if (d->seq > (int64_t(1) << 24) || d->batch > (int64_t(1) << 24) || d->heads > 1024 ||
      d->batch * d->seq > kMaxTokens)
    return fail(MCA_ERR_INVALID_ARGUMENT, "batch * seq too large");
  if (d->d_head != 64) return fail(MCA_ERR_UNSUPPORTED, "d_head must be 64 (got %lld)", (long long)d->d_head);
  const int64_t d_out = d->heads * 64;
  if (d_out % 256 != 0 || d_out > kMaxDout)
    return fail(MCA_ERR_UNSUPPORTED, "heads * 64 must be a multiple of 256 and <= %lld (got %lld)",
                (long long)kMaxDout, (long long)d_out);
  if (d->d_in > kMaxDin)
    return fail(MCA_ERR_UNSUPPORTED, "d_in must be <= %lld (got %lld)", (long long)kMaxDin, (long long)d->d_in);
  const void* opt[] = {d->seq_lens, d->r_in, d->colmax_out, d->sample_idx_out, d->sample_coef_out,
                       d->encoded_out};
  for (const void* p : opt)
    if (p && !aligned16(p)) return fail(MCA_ERR_INVALID_ARGUMENT, "optional pointers must be 16-byte aligned");
  return MCA_OK;
}

// ------------------------------------------------------------------ profiler
constexpr int kMaxRecords = 65536;

struct Profiler {
  std::mutex mu;
  std::vector<hipEvent_t> start, stop;
  std::vector<int> stage;
  int used = 0;
  ~Profiler() {
    for (auto e : start) (void)hipEventDestroy(e);
    for (auto e : stop) (void)hipEventDestroy(e);
  }
};

// Grows the event pool in chunks; returns the record slot or -1.
int prof_slot(Profiler* pr, int stage) {
  std::lock_guard<std::mutex> lk(pr->mu);
  if (pr->used >= kMaxRecords) return -1;
  if (pr->used == (int)pr->start.size()) {
    for (int i = 0; i < 256; ++i) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess) return -1;
      if (hipEventCreate(&b) != hipSuccess) {
        (void)hipEventDestroy(a);
        return -1;
      }
      pr->start.push_back(a);
      pr->stop.push_back(b);
      pr->stage.push_back(0);
    }
  }
  pr->stage[pr->used] = stage;
  return pr->used++;
}

// Launches one stage; with a profiler, its kernel carries a start and a stop event that the
// dispatch records at the kernel's start and end.
template <typename F>
mca_status run_stage(Profiler* pr, int stage, mca::FwdParams& p, F&& launch) {
  const int slot = pr ? prof_slot(pr, stage) : -1;
  p.ev_start = slot >= 0 ? pr->start[slot] : nullptr;
  p.ev_stop = slot >= 0 ? pr->stop[slot] : nullptr;
  const hipError_t e = launch();
  p.ev_start = p.ev_stop = nullptr;
  if (e != hipSuccess) {
    if (slot >= 0) {  // nothing was recorded on the slot's events: give it back
      std::lock_guard<std::mutex> lk(pr->mu);
      if (pr->used == slot + 1) --pr->used;
      else pr->stage[slot] = -1;  // a later slot is taken: collect skips this one
    }
    return fail(MCA_ERR_HIP, "stage %s launch failed: %s", mca_stage_name(stage), hipGetErrorString(e));
  }
  return MCA_OK;
}

}  // namespace

extern "C" {

const char* mca_status_string(int s) {
  switch (s) {
    case MCA_OK: return "MCA_OK";
    case MCA_ERR_INVALID_ARGUMENT: return "MCA_ERR_INVALID_ARGUMENT";
    case MCA_ERR_UNSUPPORTED: return "MCA_ERR_UNSUPPORTED";
    case MCA_ERR_WORKSPACE_TOO_SMALL: return "MCA_ERR_WORKSPACE_TOO_SMALL";
    case MCA_ERR_HIP: return "MCA_ERR_HIP";
  }
  return "MCA_ERR_UNKNOWN";
}

const char* mca_last_error(void) { return g_last_error; }

int mca_num_stages(void) { return MCA_NUM_STAGES; }

const char* mca_stage_name(int stage) {
  static const char* names[MCA_NUM_STAGES] = {"scores_colmax", "sample", "gather", "attn_out", "saturated"};
  return (stage >= 0 && stage < MCA_NUM_STAGES) ? names[stage] : "unknown";
}

mca_status mca_workspace_size(const mca_forward_desc* desc, size_t* bytes) {
  mca_status st = check_desc(desc);
  if (st != MCA_OK) return st;
  if (!bytes) return fail(MCA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  *bytes = layout_for(*desc).total;
  return ok();
}

static mca_status check_weights(int32_t dtype, int64_t d_in, int64_t d_out) {
  if (dtype != MCA_F32 && dtype != MCA_BF16) return fail(MCA_ERR_INVALID_ARGUMENT, "bad dtype %d", dtype);
  if (d_in < 1 || d_out < 1 || d_in > kMaxDin || d_out > (int64_t(1) << 20))
    return fail(MCA_ERR_INVALID_ARGUMENT, "d_in must be in 1..%lld and d_out in 1..2^20", (long long)kMaxDin);
  return MCA_OK;
}

mca_status mca_prepared_size(int32_t dtype, int64_t d_in, int64_t d_out, size_t* bytes) {
  mca_status st = check_weights(dtype, d_in, d_out);
  if (st != MCA_OK) return st;
  if (!bytes) return fail(MCA_ERR_INVALID_ARGUMENT, "bytes is NULL");
  *bytes = mca::prepared_bytes(dtype == MCA_BF16, d_in, d_out);
  return ok();
}

mca_status mca_prepare_weights(const void* W_v, int32_t dtype, int64_t d_in, int64_t d_out, void* prepared,
                               size_t prepared_bytes, void* stream) {
  if (!W_v || !prepared) return fail(MCA_ERR_INVALID_ARGUMENT, "W_v and prepared must not be NULL");
  mca_status st = check_weights(dtype, d_in, d_out);
  if (st != MCA_OK) return st;
  if (!aligned16(W_v) || !aligned16(prepared)) return fail(MCA_ERR_INVALID_ARGUMENT, "pointers must be 16-byte aligned");
  const size_t need = mca::prepared_bytes(dtype == MCA_BF16, d_in, d_out);
  if (prepared_bytes < need)
    return fail(MCA_ERR_INVALID_ARGUMENT, "prepared buffer has %zu bytes, needs %zu", prepared_bytes, need);
  hipError_t e = mca::launch_prepare(W_v, dtype == MCA_BF16, (int)d_in, (int)d_out, prepared,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(MCA_ERR_HIP, "weight preparation launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

namespace {

// Checks the tensors of a forward call and enqueues its stage kernels with `workspace` as the
// scratch memory (the caller's workspace, or the no-allocation entry's device array).
mca_status forward_impl(const mca_forward_desc* desc, const void* Q, const void* K, const void* X, const void* W_v,
                        const void* prepared, float* Y, int32_t* r, void* workspace, size_t workspace_bytes,
                        void* stream) {
  mca_status st;
  if (!Q || !K || !X || !W_v || !prepared || !Y || !r || !workspace)
    return fail(MCA_ERR_INVALID_ARGUMENT, "Q, K, X, W_v, prepared, Y, r and workspace must not be NULL");
  const void* req[] = {Q, K, X, W_v, prepared, Y, r, workspace};
  for (const void* p : req)
    if (!aligned16(p)) return fail(MCA_ERR_INVALID_ARGUMENT, "device pointers must be 16-byte aligned");
  const Layout L = layout_for(*desc);
  if (workspace_bytes < L.total)
    return fail(MCA_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);

  mca::FwdParams p{};
  p.B = (int)desc->batch;
  p.n = (int)desc->seq;
  p.H = (int)desc->heads;
  p.d_in = (int)desc->d_in;
  p.d_out = (int)(desc->heads * 64);
  p.bf16 = desc->dtype == MCA_BF16;
  p.weight_sampling = desc->sampling == MCA_SAMPLING_WEIGHT;
  p.band_half = (int)(desc->window / 2);
  p.importance = desc->importance;
  p.exact_from = desc->exact_from;
  p.qtiles = L.qtiles;
  p.nparts = L.nparts;
  p.din_pad = (int)mca::prepared_din_pad(desc->d_in);
  p.alpha = desc->alpha;
  p.seed_lo = (uint32_t)(desc->seed & 0xffffffffu);
  p.seed_hi = (uint32_t)(desc->seed >> 32);
  p.seq_lens = desc->seq_lens;
  p.r_in = desc->r_in;
  p.Q = Q;
  p.K = K;
  p.X = X;
  p.W = W_v;
  p.rownorm = static_cast<const float*>(prepared);
  p.Wt = static_cast<const char*>(prepared) + mca::prepared_wt_offset(desc->d_in);
  p.wtable = reinterpret_cast<const uint64_t*>(static_cast<const char*>(prepared) +
                                               mca::prepared_table_offset(p.bf16, desc->d_in, p.d_out));
  p.Y = Y;
  p.r = r;
  char* ws = static_cast<char*>(workspace);
  p.colmax_part = reinterpret_cast<float*>(ws + L.colmax_part);
  p.row_c = reinterpret_cast<float*>(ws + L.row_c);
  p.acol = desc->importance == MCA_IMPORTANCE_MEDIAN ? reinterpret_cast<float*>(ws + L.acol) : nullptr;
  p.Henc = ws + L.henc;
  p.list = reinterpret_cast<uint2*>(ws + L.list);
  p.ucount = reinterpret_cast<int32_t*>(ws + L.ucount);
  p.wc = mca::gather_slice_cols(p.d_in);
  // saturated tokens: inside the gather (bf16, 16-byte x chunks, d_in <= 768: the slice's
  // B operand fits in LDS next to the W_v slice), else in their own MFMA kernel
  p.sat_separate = !(p.bf16 && p.d_in % 8 == 0 && p.din_pad <= 768);
  p.gather_bps = mca::gather_blocks_per_slice(p.d_in, p.d_out);
  p.colmax_out = desc->colmax_out;
  p.idx_out = desc->sample_idx_out;
  p.coef_out = desc->sample_coef_out;
  p.enc_out = desc->encoded_out;

  hipStream_t s = static_cast<hipStream_t>(stream);
  Profiler* pr = static_cast<Profiler*>(desc->profiler);
  if ((st = run_stage(pr, MCA_STAGE_SCORES_COLMAX, p, [&] { return mca::launch_scores_colmax(p, s); })) != MCA_OK)
    return st;
  if ((st = run_stage(pr, MCA_STAGE_SAMPLE, p, [&] { return mca::launch_sample(p, s); })) != MCA_OK) return st;
  if (p.sat_separate &&
      (st = run_stage(pr, MCA_STAGE_SATURATED, p, [&] { return mca::launch_saturated(p, s); })) != MCA_OK)
    return st;
  if ((st = run_stage(pr, MCA_STAGE_GATHER, p, [&] { return mca::launch_gather(p, s); })) != MCA_OK) return st;
  if ((st = run_stage(pr, MCA_STAGE_ATTN_OUT, p, [&] { return mca::launch_attn_out(p, s); })) != MCA_OK) return st;
  return ok();
}

// ------------------------------------------------------------------ no-allocation entry
// Scratch memory of mca_attention_forward_noalloc: one array per device, held from the first
// call on that device until the process ends. Host code never passes the array's name to a
// kernel (on the host it is only a stand-in for the symbol): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and is kept per device.
constexpr size_t kScratchBytes = MCA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

mca_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(MCA_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(MCA_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!ptr) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    ptr = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!ptr) {
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ptr)
        return fail(MCA_ERR_HIP, "hipGetSymbolAddress of the scratch array failed on device %d: %s", dev,
                    hipGetErrorString(e));
      g_scratch_ptr[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return MCA_OK;
}

}  // namespace

extern "C" {

mca_status mca_attention_forward(const mca_forward_desc* desc, const void* Q, const void* K, const void* X,
                                 const void* W_v, const void* prepared, float* Y, int32_t* r, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  mca_status st = check_desc(desc);
  if (st != MCA_OK) return st;
  return forward_impl(desc, Q, K, X, W_v, prepared, Y, r, workspace, workspace_bytes, stream);
}

mca_status mca_attention_forward_noalloc(const mca_forward_desc* desc, const void* Q, const void* K, const void* X,
                                         const void* W_v, const void* prepared, float* Y, int32_t* r, void* stream) {
  mca_status st = check_desc(desc);
  if (st != MCA_OK) return st;
  if (desc->profiler)
    return fail(MCA_ERR_INVALID_ARGUMENT, "mca_attention_forward_noalloc takes no profiler (it creates HIP events)");
  const size_t need = layout_for(*desc).total;
  if (need > kScratchBytes)
    return fail(MCA_ERR_WORKSPACE_TOO_SMALL, "the call needs %zu bytes of scratch; the no-allocation entry holds %zu",
                need, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws)) != MCA_OK) return st;
  return forward_impl(desc, Q, K, X, W_v, prepared, Y, r, ws, kScratchBytes, stream);
}

mca_status mca_profiler_create(void** handle) {
  if (!handle) return fail(MCA_ERR_INVALID_ARGUMENT, "handle is NULL");
  Profiler* pr = new (std::nothrow) Profiler();
  if (!pr) return fail(MCA_ERR_INVALID_ARGUMENT, "out of host memory");
  *handle = pr;
  return ok();
}

mca_status mca_profiler_collect(void* handle, double* stage_ms, int64_t* launches, int n) {
  if (!handle || !stage_ms || !launches || n < 0 || n > MCA_NUM_STAGES)
    return fail(MCA_ERR_INVALID_ARGUMENT, "bad profiler_collect arguments");
  Profiler* pr = static_cast<Profiler*>(handle);
  std::lock_guard<std::mutex> lk(pr->mu);
  for (int i = 0; i < n; ++i) {
    stage_ms[i] = 0.0;
    launches[i] = 0;
  }
  for (int k = 0; k < pr->used; ++k) {
    if (pr->stage[k] < 0) continue;  // a launch that failed: its events were never recorded
    if (hipEventSynchronize(pr->stop[k]) != hipSuccess) return fail(MCA_ERR_HIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, pr->start[k], pr->stop[k]) != hipSuccess)
      return fail(MCA_ERR_HIP, "hipEventElapsedTime failed");
    const int st = pr->stage[k];
    if (st < n) {
      stage_ms[st] += ms;
      launches[st] += 1;
    }
  }
  pr->used = 0;
  return ok();
}

mca_status mca_profiler_destroy(void* handle) {
  delete static_cast<Profiler*>(handle);
  return ok();
}

}  // extern "C"
