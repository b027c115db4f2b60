// C-ABI entry points of libspecdec.so (declared in include/specdec.h):
// argument validation on the host, then kernel launches on the caller's
// stream.  Validation never touches the GPU, so every error path below can be
// exercised without a device.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdarg>
#include <cstdio>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "specdec.h"
#include "specdec_internal.h"

namespace {

thread_local std::string g_last_error;

specdec_status_t fail(specdec_status_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  try {
    g_last_error = buf;
  } catch (...) {   // no exception crosses the C ABI; the status code still reports the failure
  }
  return code;
}

specdec_status_t ok() {
  g_last_error.clear();
  return SPECDEC_OK;
}

}  // namespace

namespace specdec {
void set_last_error(const char* msg) {
  try {
    g_last_error = msg;
  } catch (...) {
  }
}
void clear_last_error() { g_last_error.clear(); }
}  // namespace specdec

namespace {

specdec_status_t hip_fail(hipError_t e, const char* what) {
  return fail(SPECDEC_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), static_cast<int>(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int logit_bytes(int32_t dtype) {
  switch (dtype) {
    case SPECDEC_F32: return 4;
    case SPECDEC_BF16: return 2;
    case SPECDEC_F16: return 2;
    default: return 0;
  }
}

// ---- kernel timers -------------------------------------------------------------

constexpr int kTimedKernels = 9;

struct TimedLaunch {
  int kernel;
  hipEvent_t begin, end;
};

struct Timers {
  std::mutex mu;
  int32_t mask = 0;
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> pool;
  double total_ms[kTimedKernels] = {};
  int64_t launches[kTimedKernels] = {};
};

Timers& timers() {
  static Timers t;
  return t;
}

hipEvent_t take_event(Timers& t) {
  if (!t.pool.empty()) {
    hipEvent_t e = t.pool.back();
    t.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// True when work enqueued on `stream` now would be recorded into a graph
// being captured (or when that cannot be told): such a launch is not timed,
// since its events would never be recorded by themselves.  A failed query's
// error is cleared so that the launch that follows does not report it.
bool capturing(hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
    (void)hipGetLastError();
    return true;
  }
  return cs != hipStreamCaptureStatusNone;
}

// Runs `launch` on `stream`, bracketed by timer events when timing is on and
// the stream is not being captured.
template <typename F>
hipError_t timed(int kernel, hipStream_t stream, F&& launch) {
  Timers& t = timers();
  hipEvent_t b = nullptr, e = nullptr;
  bool want = false;
  {
    std::lock_guard<std::mutex> lk(t.mu);
    want = (t.mask & (1 << kernel)) != 0;
  }
  if (want && !capturing(stream)) {
    std::lock_guard<std::mutex> lk(t.mu);
    b = take_event(t);
    e = take_event(t);
  }
  // events that end up unused go back to the pool
  auto give_back = [&] {
    std::lock_guard<std::mutex> lk(t.mu);
    try {
      if (b) t.pool.push_back(b);
      if (e) t.pool.push_back(e);
    } catch (...) {
    }
  };
  const bool timing = b && e;
  hipError_t r = timing ? hipEventRecord(b, stream) : hipSuccess;
  if (r == hipSuccess) r = launch();
  if (r == hipSuccess && timing) r = hipEventRecord(e, stream);
  if (r != hipSuccess || !timing) {
    give_back();
    return r;
  }
  std::lock_guard<std::mutex> lk(t.mu);
  try {
    t.pending.push_back({kernel, b, e});
  } catch (...) {   // the launch stands; only its timing is lost
    try {
      t.pool.push_back(b);
      t.pool.push_back(e);
    } catch (...) {
    }
  }
  return hipSuccess;
}

// ---- validation -------------------------------------------------------------------

struct Region {
  const void* p;
  int64_t bytes;
  const char* name;
};

// Every output region must be disjoint from every input region and from the
// other outputs (NULL or empty regions are skipped; inputs may overlap each
// other).  A buffer updated in place is listed once, as an output.
specdec_status_t check_disjoint(const Region* in, size_t nin, const Region* out, size_t nout) {
  auto meet = [](const Region& a, const Region& b) {
    if (!a.p || !b.p || a.bytes <= 0 || b.bytes <= 0) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
    return a0 < b0 + static_cast<uintptr_t>(b.bytes) && b0 < a0 + static_cast<uintptr_t>(a.bytes);
  };
  for (size_t o = 0; o < nout; ++o) {
    for (size_t i = 0; i < nin; ++i)
      if (meet(out[o], in[i]))
        return fail(SPECDEC_ERR_INVALID_ARGUMENT, "output %s overlaps input %s", out[o].name, in[i].name);
    for (size_t o2 = 0; o2 < o; ++o2)
      if (meet(out[o], out[o2]))
        return fail(SPECDEC_ERR_INVALID_ARGUMENT, "outputs %s and %s overlap", out[o2].name, out[o].name);
  }
  return SPECDEC_OK;
}

specdec_status_t check_disjoint(std::initializer_list<Region> inputs, std::initializer_list<Region> outputs) {
  return check_disjoint(inputs.begin(), inputs.size(), outputs.begin(), outputs.size());
}

int64_t clamp_bytes(size_t n) { return n > static_cast<size_t>(INT64_MAX) ? INT64_MAX : static_cast<int64_t>(n); }

// Greedy verification's two launches, timed as a whole (SPECDEC_KERNEL_VERIFY)
// and the vocabulary scan alone (SPECDEC_KERNEL_VERIFY_SCAN).
hipError_t verify_launches(const specdec::VerifyLaunch& p, hipStream_t st) {
  return timed(SPECDEC_KERNEL_VERIFY, st, [&] {
    const hipError_t r = timed(SPECDEC_KERNEL_VERIFY_SCAN, st, [&] { return specdec::launch_verify_scan(p, st); });
    return r != hipSuccess ? r : specdec::launch_verify_finalize(p, st);
  });
}

// Stochastic verification's launches, timed as a whole (SPECDEC_KERNEL_SAMPLE)
// and the row statistics alone (SPECDEC_KERNEL_SAMPLE_STATS).
hipError_t sample_launches(const specdec::SampleLaunch& p, hipStream_t st) {
  return timed(SPECDEC_KERNEL_SAMPLE, st, [&] {
    const hipError_t r = timed(SPECDEC_KERNEL_SAMPLE_STATS, st, [&] { return specdec::launch_sample_stats(p, st); });
    return r != hipSuccess ? r : specdec::launch_sample_finish(p, st);
  });
}

specdec_status_t check_verify_args(const void* logits, int32_t dtype, const int32_t* draft,
                                   const int32_t* pad_in, int32_t B, int32_t k, int32_t V, int32_t W_in,
                                   const int32_t* tokens, const int32_t* n_acc, const int32_t* bonus,
                                   const int32_t* pad_out, const int32_t* w_new, const void* workspace,
                                   size_t workspace_bytes, const uint32_t* dev_status) {
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (V < 1) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "V=%d must be >= 1", V);
  if (W_in < k + 1 || W_in > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "W_in=%d outside [k+1=%d, %d]", W_in, k + 1, SPECDEC_MAX_WIDTH);
  const int eb = logit_bytes(dtype);
  if (eb == 0) return fail(SPECDEC_ERR_UNSUPPORTED, "logit dtype %d not supported", dtype);
  const int64_t rows = static_cast<int64_t>(B) * (k + 1);
  if (rows > SPECDEC_MAX_ROWS) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B*(k+1)=%lld exceeds %d", (long long)rows, SPECDEC_MAX_ROWS);
  if (B == 0) return SPECDEC_OK;
  if (!logits || !pad_in || !tokens || !n_acc || !pad_out || !w_new || (k > 0 && !draft))
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL tensor pointer (logits, draft, pad_in, tokens, n_acc, pad_out, w_new)");
  if (!aligned(logits, eb)) return fail(SPECDEC_ERR_UNSUPPORTED, "logits not aligned to %d bytes", eb);
  const void* i32s[] = {draft, pad_in, tokens, n_acc, bonus, pad_out, w_new};
  for (const void* p : i32s)
    if (p && !aligned(p, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  {
    const int64_t b4 = 4 * static_cast<int64_t>(B);
    specdec_status_t d = check_disjoint(
        {{logits, rows * V * eb, "logits"}, {draft, b4 * k, "draft"}, {pad_in, b4, "pad_in"}},
        {{tokens, b4 * (k + 1), "tokens"}, {n_acc, b4, "n_acc"}, {bonus, b4, "bonus"}, {pad_out, b4, "pad_out"},
         {w_new, 4, "w_new"}, {workspace, clamp_bytes(workspace_bytes), "workspace"},
         {dev_status, 4, "dev_status"}});
    if (d) return d;
  }
  const int64_t chunk = specdec::verify_chunk_elems(rows, V);
  const int64_t blocks = rows * ((V + chunk - 1) / chunk);
  if (blocks * specdec::kThreads > 0xFFFFFFFFLL) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "logits too large for one launch");
  const size_t need = specdec_workspace_bytes(B, k, V);
  if (!workspace) return fail(SPECDEC_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (!aligned(workspace, 8)) return fail(SPECDEC_ERR_WORKSPACE, "workspace not 8-byte aligned");
  if (workspace_bytes < need)
    return fail(SPECDEC_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  return SPECDEC_OK;
}

specdec_status_t check_kv(const specdec_kv_t* kv, const char* name) {
  if (!kv) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s descriptor is NULL", name);
  if (kv->L < 0 || kv->B < 0 || kv->H < 0) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s has a negative dimension", name);
  if (kv->D <= 0 || kv->D > SPECDEC_MAX_D) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s D=%d outside [1,%d]", name, kv->D, SPECDEC_MAX_D);
  if (kv->D % 8 != 0) return fail(SPECDEC_ERR_UNSUPPORTED, "%s D=%d: rows of D bf16 must be whole 16-byte vectors", name, kv->D);
  if (kv->cap < 0 || kv->cap > SPECDEC_MAX_WIDTH) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s cap=%lld out of range", name, (long long)kv->cap);
  const int64_t spans = static_cast<int64_t>(kv->L) * 2 * kv->B * kv->H;
  if (spans > 0x7FFFFFFFLL) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s has too many spans", name);
  if (spans > 0 && kv->cap > 0) {
    if (!kv->data) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s data is NULL", name);
    if (!aligned(kv->data, 16)) return fail(SPECDEC_ERR_UNSUPPORTED, "%s data not 16-byte aligned", name);
  }
  return SPECDEC_OK;
}

int64_t kv_bytes(const specdec_kv_t* kv) {
  return static_cast<int64_t>(kv->L) * 2 * kv->B * kv->H * kv->cap * kv->D * 2;
}

specdec_status_t check_realign_args(const specdec_kv_t* src, const specdec_kv_t* dst, int32_t k, int32_t W_in,
                                    const int32_t* pad_in, const int32_t* n_acc, const int32_t* w_new,
                                    bool* in_place) {
  specdec_status_t s = check_kv(src, "src");
  if (s) return s;
  s = check_kv(dst, "dst");
  if (s) return s;
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (W_in < k + 1 || W_in > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "W_in=%d outside [k+1=%d, %d]", W_in, k + 1, SPECDEC_MAX_WIDTH);
  if (src->L != dst->L || src->B != dst->B || src->H != dst->H || src->D != dst->D)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "src and dst shapes differ");
  const int64_t spans = static_cast<int64_t>(src->L) * 2 * src->B * src->H;
  *in_place = false;
  if (spans == 0) return SPECDEC_OK;
  if (src->cap < W_in) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "src cap=%lld < W_in=%d", (long long)src->cap, W_in);
  if (dst->cap < W_in) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "dst cap=%lld < W_in=%d", (long long)dst->cap, W_in);
  if (!pad_in || !n_acc || !w_new) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL pad_in / n_acc / w_new");
  if (!aligned(pad_in, 4) || !aligned(n_acc, 4) || !aligned(w_new, 4))
    return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src->data), d0 = reinterpret_cast<uintptr_t>(dst->data);
  const uintptr_t s1 = s0 + static_cast<uintptr_t>(kv_bytes(src)), d1 = d0 + static_cast<uintptr_t>(kv_bytes(dst));
  if (s0 == d0) {
    if (src->cap != dst->cap) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "in place needs src cap == dst cap");
    *in_place = true;
  } else if (s0 < d1 && d0 < s1) {
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "src and dst overlap without being the same cache");
  }
  if (spans > 0xFFFFFFFFLL) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "too many spans");
  return SPECDEC_OK;
}

specdec_status_t check_token_args(const int32_t* s_in, int64_t s_in_stride, const int32_t* s_out,
                                  int64_t s_out_stride, int32_t B, int32_t k, int32_t W_in) {
  if (B == 0) return SPECDEC_OK;
  if (!s_in || !s_out) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL token row");
  if (!aligned(s_in, 4) || !aligned(s_out, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "token row not 4-byte aligned");
  if (s_in_stride < static_cast<int64_t>(W_in) - k || s_in_stride > SPECDEC_MAX_WIDTH + 1)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "s_in_stride=%lld < W_in-k=%d", (long long)s_in_stride, W_in - k);
  if (s_out_stride < static_cast<int64_t>(W_in) + 1 || s_out_stride > SPECDEC_MAX_WIDTH + 1)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "s_out_stride=%lld < W_in+1=%d", (long long)s_out_stride, W_in + 1);
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(s_in), b0 = reinterpret_cast<uintptr_t>(s_out);
  const uintptr_t a1 = a0 + static_cast<uintptr_t>(B) * s_in_stride * 4, b1 = b0 + static_cast<uintptr_t>(B) * s_out_stride * 4;
  if (a0 == b0) {
    if (s_in_stride != s_out_stride) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "in-place token row needs equal strides");
  } else if (a0 < b1 && b0 < a1) {
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "token rows overlap without being the same buffer");
  }
  return SPECDEC_OK;
}

specdec_status_t check_posmask_args(const int32_t* pad_out, const int32_t* w_new, int32_t B, int32_t k,
                                    const int64_t* pos, const uint8_t* mask, int64_t pm_cap,
                                    const uint32_t* dev_status) {
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (pm_cap < k + 1 || pm_cap > SPECDEC_MAX_WIDTH + SPECDEC_MAX_K + 1)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pm_cap=%lld out of range", (long long)pm_cap);
  if (B == 0) return SPECDEC_OK;
  if (!pad_out || !w_new || !pos || !mask) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL pad_out / w_new / pos / mask");
  if (!aligned(pos, 8)) return fail(SPECDEC_ERR_UNSUPPORTED, "pos not 8-byte aligned");
  if (!aligned(pad_out, 4) || !aligned(w_new, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  const int64_t n = static_cast<int64_t>(B) * pm_cap;
  return check_disjoint({{pad_out, 4 * static_cast<int64_t>(B), "pad_out"}, {w_new, 4, "w_new"}},
                        {{pos, 8 * n, "pos"}, {mask, n, "mask"}, {dev_status, 4, "dev_status"}});
}


specdec_status_t check_sample_args(const void* logits, const void* draft_logits, int32_t dtype, const int32_t* draft,
                                   const int32_t* pad_in, const float* u_accept, const float* u_sample,
                                   float temperature, int32_t B, int32_t k, int32_t V, int32_t W_in,
                                   const int32_t* tokens, const int32_t* n_acc, const int32_t* bonus,
                                   const int32_t* pad_out, const int32_t* w_new, const void* workspace,
                                   size_t workspace_bytes, const uint32_t* dev_status, float* c_out) {
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (V < 1 || V > SPECDEC_MAX_SAMPLE_V)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "V=%d outside [1, %d]", V, SPECDEC_MAX_SAMPLE_V);
  if (W_in < k + 1 || W_in > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "W_in=%d outside [k+1=%d, %d]", W_in, k + 1, SPECDEC_MAX_WIDTH);
  const int eb = logit_bytes(dtype);
  if (eb == 0) return fail(SPECDEC_ERR_UNSUPPORTED, "logit dtype %d not supported", dtype);
  const double c = 1.4426950408889634 / static_cast<double>(temperature);
  if (!(temperature > 0.0f) || !std::isfinite(temperature) || !std::isfinite(static_cast<float>(c)))
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "temperature %g must be finite and > 0 (with log2(e)/T finite)",
                static_cast<double>(temperature));
  *c_out = static_cast<float>(c);
  const int64_t rows = static_cast<int64_t>(B) * (2 * k + 1);
  if (rows > SPECDEC_MAX_ROWS)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B*(2k+1)=%lld exceeds %d", (long long)rows, SPECDEC_MAX_ROWS);
  if (B == 0) return SPECDEC_OK;
  if (!logits || !pad_in || !u_sample || !tokens || !n_acc || !pad_out || !w_new ||
      (k > 0 && (!draft || !draft_logits || !u_accept)))
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL tensor pointer");
  if (!aligned(logits, eb) || (draft_logits && !aligned(draft_logits, eb)))
    return fail(SPECDEC_ERR_UNSUPPORTED, "logits not aligned to %d bytes", eb);
  const void* w4[] = {draft, pad_in, u_accept, u_sample, tokens, n_acc, bonus, pad_out, w_new, dev_status};
  for (const void* q : w4)
    if (q && !aligned(q, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "4-byte tensor not 4-byte aligned");
  {
    const int64_t b4 = 4 * static_cast<int64_t>(B);
    const int64_t lb = static_cast<int64_t>(B) * V * eb;
    specdec_status_t d = check_disjoint(
        {{logits, lb * (k + 1), "logits"}, {draft_logits, lb * k, "draft_logits"}, {draft, b4 * k, "draft"},
         {pad_in, b4, "pad_in"}, {u_accept, b4 * k, "u_accept"}, {u_sample, b4, "u_sample"}},
        {{tokens, b4 * (k + 1), "tokens"}, {n_acc, b4, "n_acc"}, {bonus, b4, "bonus"}, {pad_out, b4, "pad_out"},
         {w_new, 4, "w_new"}, {workspace, clamp_bytes(workspace_bytes), "workspace"},
         {dev_status, 4, "dev_status"}});
    if (d) return d;
  }
  const int64_t blocks = rows * specdec::sample_chunks(rows, V);
  if (blocks * 256 > 0xFFFFFFFFLL) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "logits too large for one launch");
  const size_t need = specdec_sample_workspace_bytes(B, k, V);
  if (!workspace) return fail(SPECDEC_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", need);
  if (!aligned(workspace, 8)) return fail(SPECDEC_ERR_WORKSPACE, "workspace not 8-byte aligned");
  if (workspace_bytes < need)
    return fail(SPECDEC_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  return SPECDEC_OK;
}

// Checks shared by the fused steps after their verification arguments.
specdec_status_t check_step_rest(int32_t B, int32_t k, int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                                 const int32_t* pad_in, const int32_t* n_acc, const int32_t* pad_out,
                                 const int32_t* w_new, const int64_t* pos, const uint8_t* mask, int64_t pm_cap,
                                 const int32_t* s_in, int64_t s_in_stride, const int32_t* s_out,
                                 int64_t s_out_stride, const uint32_t* dev_status, bool* in_place) {
  specdec_status_t s = check_realign_args(src, dst, k, W_in, pad_in, n_acc, w_new, in_place);
  if (s) return s;
  if (src->B != B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "cache rows B=%d differ from logits rows B=%d", src->B, B);
  s = check_posmask_args(pad_out, w_new, B, k, pos, mask, pm_cap, dev_status);
  if (s) return s;
  if (B > 0 && pm_cap < static_cast<int64_t>(W_in) + k + 1)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pm_cap=%lld < W_in+k+1=%d", (long long)pm_cap, W_in + k + 1);
  if (s_in || s_out) {
    s = check_token_args(s_in, s_in_stride, s_out, s_out_stride, B, k, W_in);
    if (s) return s;
  }
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  return SPECDEC_OK;
}

// Every buffer of a fused step against every output: the verification inputs,
// the source cache and token row, then the verification outputs, workspace,
// position ids / mask, destination cache and token row and the status word.
// A cache or token row realigned in place is listed once, as an output.
struct StepInputs {
  const void* logits;
  int64_t logit_bytes;            // target logits [B][k+1][V]
  const void* draft_logits;       // [B][k][V] (stochastic verification) or NULL
  int64_t draft_logit_bytes;
  const int32_t* draft;
  const int32_t* pad_in;
  const float* u_accept;          // [B][k] or NULL
  const float* u_sample;          // [B] or NULL
};

specdec_status_t check_step_disjoint(const StepInputs& v, int32_t B, int32_t k, const specdec_kv_t* src,
                                     const specdec_kv_t* dst, bool in_place, const int32_t* tokens,
                                     const int32_t* n_acc, const int32_t* bonus, const int32_t* pad_out,
                                     const int32_t* w_new, const void* workspace, size_t workspace_bytes,
                                     const int64_t* pos, const uint8_t* mask, int64_t pm_cap, const int32_t* s_in,
                                     int64_t s_in_stride, const int32_t* s_out, int64_t s_out_stride,
                                     const uint32_t* dev_status) {
  const int64_t b4 = 4 * static_cast<int64_t>(B), pm = static_cast<int64_t>(B) * pm_cap;
  const bool tok_in_place = s_in == s_out;
  const Region in[] = {{v.logits, v.logit_bytes, "logits"},
                       {v.draft_logits, v.draft_logit_bytes, "draft_logits"},
                       {v.draft, b4 * k, "draft"},
                       {v.pad_in, b4, "pad_in"},
                       {v.u_accept, b4 * k, "u_accept"},
                       {v.u_sample, b4, "u_sample"},
                       {in_place ? nullptr : src->data, kv_bytes(src), "src cache"},
                       {tok_in_place ? nullptr : s_in, s_in ? b4 * s_in_stride : 0, "s_in"}};
  const Region out[] = {{tokens, b4 * (k + 1), "tokens"},
                        {n_acc, b4, "n_acc"},
                        {bonus, b4, "bonus"},
                        {pad_out, b4, "pad_out"},
                        {w_new, 4, "w_new"},
                        {workspace, clamp_bytes(workspace_bytes), "workspace"},
                        {pos, 8 * pm, "pos"},
                        {mask, pm, "mask"},
                        {dst->data, kv_bytes(dst), "dst cache"},
                        {s_out, s_out ? b4 * s_out_stride : 0, "s_out"},
                        {dev_status, 4, "dev_status"}};
  return check_disjoint(in, sizeof(in) / sizeof(in[0]), out, sizeof(out) / sizeof(out[0]));
}

// The realignment launch of a fused step (cache, position ids / mask, token
// row), then the optional host copy of the new width.
specdec_status_t step_realign(int32_t k, int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                              bool in_place, const int32_t* pad_in, const int32_t* tokens, const int32_t* n_acc,
                              const int32_t* pad_out, const int32_t* w_new, int64_t* pos, uint8_t* mask,
                              int64_t pm_cap, const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                              int64_t s_out_stride, int32_t pad_id, uint32_t* dev_status, int32_t* w_new_host,
                              hipStream_t st, uint32_t* clear_words = nullptr, uint32_t clear_count = 0,
                              const int32_t* order = nullptr) {
  specdec::RealignLaunch rp{};
  rp.clear_words = clear_words;
  rp.clear_count = clear_count;
  rp.order = order;
  rp.src = src->data;
  rp.dst = dst->data;
  rp.src_cap = src->cap;
  rp.dst_cap = dst->cap;
  rp.L = src->L;
  rp.B = src->B;
  rp.H = src->H;
  rp.D = src->D;
  rp.k = k;
  rp.W_in = W_in;
  rp.pad_in = pad_in;
  rp.n_acc = n_acc;
  rp.w_new = w_new;
  rp.dev_status = dev_status;
  rp.in_place = in_place;
  rp.pos = pos;
  rp.mask = mask;
  rp.pm_cap = pm_cap;
  rp.pad_out = pad_out;
  rp.s_in = s_in;
  rp.s_out = s_out;
  rp.s_in_stride = s_in_stride;
  rp.s_out_stride = s_out_stride;
  rp.tokens = tokens;
  rp.pad_id = pad_id;
  hipError_t e = timed(SPECDEC_KERNEL_REALIGN, st, [&] { return specdec::launch_realign(rp, st); });
  if (e != hipSuccess) return hip_fail(e, "realign launch");
  if (w_new_host) {
    e = hipMemcpyAsync(w_new_host, w_new, sizeof(int32_t), hipMemcpyDeviceToHost, st);
    if (e != hipSuccess) return hip_fail(e, "w_new copy");
    e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  }
  return ok();
}

bool ranges_overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + static_cast<uintptr_t>(bbytes) && b0 < a0 + static_cast<uintptr_t>(abytes);
}

// Common checks of the pool / batch pair of a gather or write-back.
specdec_status_t check_pool_pair(const specdec_kv_t* pool, const specdec_kv_t* batch, int32_t B, int32_t Lb,
                                 int32_t k, int64_t batch_cap_min, const int32_t* lens, const int32_t* slots) {
  specdec_status_t s = check_kv(pool, "pool");
  if (s) return s;
  s = check_kv(batch, "batch");
  if (s) return s;
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (Lb < 0 || Lb > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "Lb=%d outside [0,%d]", Lb, SPECDEC_MAX_WIDTH);
  if (batch->B != B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch has %d rows, B=%d", batch->B, B);
  if (pool->L != batch->L || pool->H != batch->H || pool->D != batch->D)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pool and batch shapes differ");
  if (B == 0) return SPECDEC_OK;
  if (pool->B < 1) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "the pool has no slot");
  if (!lens || !slots) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL lens / slots");
  if (!aligned(lens, 4) || !aligned(slots, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  const int64_t spans = static_cast<int64_t>(batch->L) * 2 * B * batch->H;
  if (spans > 0) {
    if (batch->cap < batch_cap_min)
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch cap=%lld < %lld", (long long)batch->cap, (long long)batch_cap_min);
    if (pool->cap > 0 && batch->cap > 0 && ranges_overlap(pool->data, kv_bytes(pool), batch->data, kv_bytes(batch)))
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pool and batch caches overlap");
  }
  return SPECDEC_OK;
}

specdec_status_t check_stride(int64_t stride, int64_t need, const char* name) {
  if (stride < need || stride > static_cast<int64_t>(SPECDEC_MAX_WIDTH) + SPECDEC_MAX_K + 2)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "%s=%lld outside [%lld, %lld]", name, (long long)stride, (long long)need,
                (long long)SPECDEC_MAX_WIDTH + SPECDEC_MAX_K + 2);
  return SPECDEC_OK;
}

}  // namespace

extern "C" {

int32_t specdec_abi_version(void) { return SPECDEC_ABI_VERSION; }

const char* specdec_last_error(void) { return g_last_error.c_str(); }

size_t specdec_workspace_bytes(int32_t B, int32_t k, int32_t V) {
  if (B < 0 || B > SPECDEC_MAX_B || k < 0 || k > SPECDEC_MAX_K || V < 1) return 0;
  // header, partial maxima, then the in-place realignment order
  return static_cast<size_t>(specdec::order_offset(B, k, V) + specdec::order_bytes(B));
}

specdec_status_t specdec_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (workspace_bytes == 0) return ok();
  if (!workspace) return fail(SPECDEC_ERR_WORKSPACE, "workspace is NULL");
  hipError_t e = specdec::launch_zero(workspace, workspace_bytes, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "workspace clear");
  return ok();
}

specdec_status_t specdec_verify_greedy(const void* logits, int32_t dtype, const int32_t* draft,
                                       const int32_t* pad_in, int32_t B, int32_t k, int32_t V, int32_t W_in,
                                       int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                                       int32_t* w_new, void* workspace, size_t workspace_bytes,
                                       uint32_t* dev_status, void* stream) {
  specdec_status_t s = check_verify_args(logits, dtype, draft, pad_in, B, k, V, W_in, tokens, n_acc, bonus,
                                         pad_out, w_new, workspace, workspace_bytes, dev_status);
  if (s) return s;
  if (B == 0) return ok();
  specdec::VerifyLaunch p{logits, dtype, draft, pad_in, B, k, V, W_in, tokens, n_acc,
                          bonus, pad_out, w_new, workspace, dev_status};
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = verify_launches(p, st);
  if (e != hipSuccess) return hip_fail(e, "verify launch");
  return ok();
}

size_t specdec_sample_workspace_bytes(int32_t B, int32_t k, int32_t V) {
  if (B < 0 || B > SPECDEC_MAX_B || k < 0 || k > SPECDEC_MAX_K || V < 1 || V > SPECDEC_MAX_SAMPLE_V) return 0;
  const int64_t rows = static_cast<int64_t>(B) * (2 * k + 1);
  // chunk statistics of every row, then per (sequence, chunk) the two last
  // indices and per (sequence, chunk, tile of 2048 logits) the two masses
  const int64_t chunks = specdec::sample_chunks(rows, V);
  const int64_t mc = specdec::sample_mass_chunk_elems(B, V);
  const int64_t mchunks = (V + mc - 1) / mc;
  const int64_t tiles = (mc + 2047) / 2048;
  return specdec::kWsHeaderBytes + static_cast<size_t>(B) * 16u +
         static_cast<size_t>(rows * chunks + B * mchunks * (1 + tiles)) * 8u;
}

specdec_status_t specdec_verify_sample(const void* logits, const void* draft_logits, int32_t dtype,
                                       const int32_t* draft, const int32_t* pad_in, const float* u_accept,
                                       const float* u_sample, float temperature, int32_t B, int32_t k, int32_t V,
                                       int32_t W_in, int32_t* tokens, int32_t* n_acc, int32_t* bonus,
                                       int32_t* pad_out, int32_t* w_new, void* workspace, size_t workspace_bytes,
                                       uint32_t* dev_status, void* stream) {
  float c = 0.0f;
  specdec_status_t s = check_sample_args(logits, draft_logits, dtype, draft, pad_in, u_accept, u_sample, temperature, B,
                                         k, V, W_in, tokens, n_acc, bonus, pad_out, w_new, workspace, workspace_bytes,
                                         dev_status, &c);
  if (s || B == 0) return s ? s : ok();
  specdec::SampleLaunch p{logits, draft_logits, dtype, draft, pad_in, u_accept, u_sample, c,
                          B, k, V, W_in, tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status};
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = sample_launches(p, st);
  if (e != hipSuccess) return hip_fail(e, "stochastic verify launch");
  return ok();
}

specdec_status_t specdec_realign_kv(const specdec_kv_t* src, const specdec_kv_t* dst, int32_t k, int32_t W_in,
                                    const int32_t* pad_in, const int32_t* n_acc, const int32_t* w_new,
                                    uint32_t* dev_status, void* stream) {
  bool in_place = false;
  specdec_status_t s = check_realign_args(src, dst, k, W_in, pad_in, n_acc, w_new, &in_place);
  if (s) return s;
  if (static_cast<int64_t>(src->L) * src->B * src->H == 0) return ok();
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  {
    const int64_t b4 = 4 * static_cast<int64_t>(src->B);
    s = check_disjoint({{pad_in, b4, "pad_in"}, {n_acc, b4, "n_acc"}, {w_new, 4, "w_new"},
                        {in_place ? nullptr : src->data, kv_bytes(src), "src cache"}},
                       {{dst->data, kv_bytes(dst), "dst cache"}, {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  specdec::RealignLaunch p{};
  p.src = src->data;
  p.dst = dst->data;
  p.src_cap = src->cap;
  p.dst_cap = dst->cap;
  p.L = src->L;
  p.B = src->B;
  p.H = src->H;
  p.D = src->D;
  p.k = k;
  p.W_in = W_in;
  p.pad_in = pad_in;
  p.n_acc = n_acc;
  p.w_new = w_new;
  p.dev_status = dev_status;
  p.in_place = in_place;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(SPECDEC_KERNEL_REALIGN, st, [&] { return specdec::launch_realign(p, st); });
  if (e != hipSuccess) return hip_fail(e, "realign launch");
  return ok();
}

specdec_status_t specdec_build_posmask(const int32_t* pad_out, const int32_t* w_new, int32_t B, int32_t k,
                                       int64_t* pos, uint8_t* mask, int64_t pm_cap, uint32_t* dev_status,
                                       void* stream) {
  specdec_status_t s = check_posmask_args(pad_out, w_new, B, k, pos, mask, pm_cap, dev_status);
  if (s) return s;
  if (B == 0) return ok();
  specdec::PosmaskLaunch p{pad_out, w_new, B, k, pos, mask, pm_cap, pm_cap, dev_status};
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(SPECDEC_KERNEL_POSMASK, st, [&] { return specdec::launch_posmask(p, st); });
  if (e != hipSuccess) return hip_fail(e, "posmask launch");
  return ok();
}

specdec_status_t specdec_realign_tokens(const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                                        int64_t s_out_stride, const int32_t* tokens, const int32_t* pad_in,
                                        const int32_t* n_acc, const int32_t* w_new, int32_t B, int32_t k,
                                        int32_t W_in, int32_t pad_id, uint32_t* dev_status, void* stream) {
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (W_in < k + 1 || W_in > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "W_in=%d outside [k+1=%d, %d]", W_in, k + 1, SPECDEC_MAX_WIDTH);
  specdec_status_t s = check_token_args(s_in, s_in_stride, s_out, s_out_stride, B, k, W_in);
  if (s) return s;
  if (B == 0) return ok();
  if (!tokens || !pad_in || !n_acc || !w_new) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL tokens / pad_in / n_acc / w_new");
  if (!aligned(tokens, 4) || !aligned(pad_in, 4) || !aligned(n_acc, 4) || !aligned(w_new, 4))
    return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  {
    const int64_t b4 = 4 * static_cast<int64_t>(B);
    s = check_disjoint({{tokens, b4 * (k + 1), "tokens"}, {pad_in, b4, "pad_in"}, {n_acc, b4, "n_acc"},
                        {w_new, 4, "w_new"}, {s_in == s_out ? nullptr : s_in, b4 * s_in_stride, "s_in"}},
                       {{s_out, b4 * s_out_stride, "s_out"}, {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  specdec::RealignLaunch p{};
  p.B = B;
  p.k = k;
  p.W_in = W_in;
  p.pad_in = pad_in;
  p.n_acc = n_acc;
  p.w_new = w_new;
  p.dev_status = dev_status;
  p.s_in = s_in;
  p.s_out = s_out;
  p.s_in_stride = s_in_stride;
  p.s_out_stride = s_out_stride;
  p.tokens = tokens;
  p.pad_id = pad_id;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = specdec::launch_tokens(p, st);
  if (e != hipSuccess) return hip_fail(e, "token row launch");
  return ok();
}

namespace {

// The fused step.  With `fused_counts` (library scratch whose B + 1 counts are
// zero) verification runs as one launch and the realignment launch zeroes
// the counts again; otherwise verification is the scan and merge launches on
// the caller's workspace.
specdec_status_t step_greedy(const void* logits, int32_t dtype, const int32_t* draft, const int32_t* pad_in, int32_t B,
                             int32_t k, int32_t V, int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                             int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out, int32_t* w_new,
                             int64_t* pos, uint8_t* mask, int64_t pm_cap, const int32_t* s_in, int64_t s_in_stride,
                             int32_t* s_out, int64_t s_out_stride, int32_t pad_id, void* workspace,
                             size_t workspace_bytes, uint32_t* dev_status, int32_t* w_new_host, void* stream,
                             uint32_t* fused_counts, specdec_status_t (*before_launch)(void*) = nullptr,
                             void* before_launch_ctx = nullptr) {
  specdec_status_t s = check_verify_args(logits, dtype, draft, pad_in, B, k, V, W_in, tokens, n_acc, bonus,
                                         pad_out, w_new, workspace, workspace_bytes, dev_status);
  if (s) return s;
  bool in_place = false;
  s = check_step_rest(B, k, W_in, src, dst, pad_in, n_acc, pad_out, w_new, pos, mask, pm_cap, s_in, s_in_stride, s_out,
                      s_out_stride, dev_status, &in_place);
  if (s) return s;
  {
    const StepInputs v{logits, static_cast<int64_t>(B) * (k + 1) * V * logit_bytes(dtype), nullptr, 0, draft, pad_in,
                       nullptr, nullptr};
    s = check_step_disjoint(v, B, k, src, dst, in_place, tokens, n_acc, bonus, pad_out, w_new, workspace,
                            workspace_bytes, pos, mask, pm_cap, s_in, s_in_stride, s_out, s_out_stride, dev_status);
    if (s) return s;
  }
  if (B == 0) return ok();
  // every check has passed: only now may anything be enqueued
  if (before_launch) {
    s = before_launch(before_launch_ctx);
    if (s) return s;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  specdec::VerifyLaunch vp{logits, dtype, draft, pad_in, B, k, V, W_in, tokens, n_acc,
                           bonus, pad_out, w_new, workspace, dev_status};
  // in place, the merge launch also writes the order the walk takes the rows in
  vp.write_order = in_place && !fused_counts;
  const int32_t* order =
      vp.write_order ? reinterpret_cast<const int32_t*>(static_cast<const char*>(workspace) + specdec::order_offset(B, k, V))
                     : nullptr;
  hipError_t e = fused_counts ? timed(SPECDEC_KERNEL_VERIFY, st, [&] {
    return timed(SPECDEC_KERNEL_VERIFY_SCAN, st, [&] { return specdec::launch_verify_fused(vp, fused_counts, st); });
  })
                              : verify_launches(vp, st);
  if (e != hipSuccess) return hip_fail(e, "verify launch");
  return step_realign(k, W_in, src, dst, in_place, pad_in, tokens, n_acc, pad_out, w_new, pos, mask, pm_cap, s_in,
                      s_in_stride, s_out, s_out_stride, pad_id, dev_status, w_new_host, st, fused_counts,
                      fused_counts ? static_cast<uint32_t>(B) + 1u : 0u, order);
}

}  // namespace

specdec_status_t specdec_step(const void* logits, int32_t dtype, const int32_t* draft, const int32_t* pad_in,
                              int32_t B, int32_t k, int32_t V, int32_t W_in, const specdec_kv_t* src,
                              const specdec_kv_t* dst, int32_t* tokens, int32_t* n_acc, int32_t* bonus,
                              int32_t* pad_out, int32_t* w_new, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                              const int32_t* s_in, int64_t s_in_stride, int32_t* s_out, int64_t s_out_stride,
                              int32_t pad_id, void* workspace, size_t workspace_bytes, uint32_t* dev_status,
                              int32_t* w_new_host, void* stream) {
  return step_greedy(logits, dtype, draft, pad_in, B, k, V, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new, pos,
                     mask, pm_cap, s_in, s_in_stride, s_out, s_out_stride, pad_id, workspace, workspace_bytes,
                     dev_status, w_new_host, stream, nullptr);
}

// ---- specdec_step_noalloc: the fused step on library-owned scratch -----------
//
// The step's scratch lives in `scratch`, a file-scope device array.  Each
// device the library runs on holds its own copy until the process ends.  In
// host code the name only identifies the symbol (it is not a device
// address): the device address of each device's copy is taken once, with
// that device current, by hipGetSymbolAddress, and only that address is ever
// handed to a kernel.  Layout: the partial maxima of the two-launch
// verification from the start, and, in the last kCountsBytes, the completion
// counts of the one-launch verification, zeroed by a kernel before the
// device's first step that passes its argument checks and zeroed again by
// every step's realignment launch.
static __device__ __align__(256) unsigned char scratch[SPECDEC_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kCountsBytes = 64 * 1024;   // 2 * kMaxFusedVerifyRows + 1 words and then some
static_assert((2 * specdec::kMaxFusedVerifyRows + 1) * 4 <= static_cast<int64_t>(kCountsBytes), "counts fit");
constexpr size_t kPartialBytes = SPECDEC_NOALLOC_SCRATCH_BYTES - kCountsBytes;
constexpr int kMaxScratchDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices] = {};
bool g_scratch_counts_clear[kMaxScratchDevices] = {};

struct ScratchUse {
  int dev;
  void* addr;
  hipStream_t stream;
};

// Device address of the current device's scratch (a query: nothing is
// enqueued); the stream, when given, must belong to that device.
specdec_status_t scratch_address(hipStream_t stream, ScratchUse* u) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (stream) {
    int sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if (sdev != dev)
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "stream belongs to device %d, the current device is %d", sdev, dev);
  }
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(SPECDEC_ERR_UNSUPPORTED, "device index %d beyond the scratch table (%d)", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* addr = nullptr;
    e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!addr) return fail(SPECDEC_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[dev] = addr;
  }
  *u = ScratchUse{dev, g_scratch_addr[dev], stream};
  return SPECDEC_OK;
}

// Run by the step once its arguments have passed every check: on the
// device's first such step, clears the one-launch verification's counts on
// the step's stream, ahead of its kernels (a kernel, not a memset, so that a
// first call under graph capture records no memset node).
specdec_status_t scratch_first_use(void* ctx) {
  const ScratchUse* u = static_cast<const ScratchUse*>(ctx);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_counts_clear[u->dev]) return SPECDEC_OK;
  const hipError_t e = specdec::launch_zero(static_cast<char*>(u->addr) + kPartialBytes, kCountsBytes, u->stream);
  if (e != hipSuccess) return hip_fail(e, "scratch count clear");
  g_scratch_counts_clear[u->dev] = true;
  return SPECDEC_OK;
}

}  // namespace

specdec_status_t specdec_step_noalloc(const void* logits, int32_t dtype, const int32_t* draft, const int32_t* pad_in,
                                      int32_t B, int32_t k, int32_t V, int32_t W_in, const specdec_kv_t* src,
                                      const specdec_kv_t* dst, int32_t* tokens, int32_t* n_acc, int32_t* bonus,
                                      int32_t* pad_out, int32_t* w_new, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                      const int32_t* s_in, int64_t s_in_stride, int32_t* s_out, int64_t s_out_stride,
                                      int32_t pad_id, uint32_t* dev_status, int32_t* w_new_host, void* stream) {
  void* ws = nullptr;
  size_t ws_bytes = 0;
  uint32_t* counts = nullptr;
  ScratchUse use{};
  if (B > 0) {
    const bool fused = specdec::verify_fused_fits(B, k, V, dtype);
    const size_t need = specdec_workspace_bytes(B, k, V);
    if (!fused && need > kPartialBytes)
      return fail(SPECDEC_ERR_WORKSPACE,
                  "specdec_step_noalloc: verification of B=%d, k=%d, V=%d needs %zu bytes of scratch, more than the "
                  "library's %zu of %d (use specdec_step with a workspace)",
                  B, k, V, need, kPartialBytes, SPECDEC_NOALLOC_SCRATCH_BYTES);
    const specdec_status_t s = scratch_address(static_cast<hipStream_t>(stream), &use);
    if (s) return s;
    ws = use.addr;
    ws_bytes = kPartialBytes;
    if (fused) counts = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + kPartialBytes);
  }
  return step_greedy(logits, dtype, draft, pad_in, B, k, V, W_in, src, dst, tokens, n_acc, bonus, pad_out, w_new, pos,
                     mask, pm_cap, s_in, s_in_stride, s_out, s_out_stride, pad_id, ws, ws_bytes, dev_status,
                     w_new_host, stream, counts, B > 0 ? scratch_first_use : nullptr, &use);
}

specdec_status_t specdec_step_sample(const void* logits, const void* draft_logits, int32_t dtype,
                                     const int32_t* draft, const int32_t* pad_in, const float* u_accept,
                                     const float* u_sample, float temperature, int32_t B, int32_t k, int32_t V,
                                     int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                                     int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                                     int32_t* w_new, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                     const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                                     int64_t s_out_stride, int32_t pad_id, void* workspace,
                                     size_t workspace_bytes, uint32_t* dev_status, int32_t* w_new_host,
                                     void* stream) {
  float c = 0.0f;
  specdec_status_t s = check_sample_args(logits, draft_logits, dtype, draft, pad_in, u_accept, u_sample, temperature, B,
                                         k, V, W_in, tokens, n_acc, bonus, pad_out, w_new, workspace, workspace_bytes,
                                         dev_status, &c);
  if (s) return s;
  bool in_place = false;
  s = check_step_rest(B, k, W_in, src, dst, pad_in, n_acc, pad_out, w_new, pos, mask, pm_cap, s_in, s_in_stride, s_out,
                      s_out_stride, dev_status, &in_place);
  if (s) return s;
  {
    const int64_t lb = static_cast<int64_t>(B) * V * logit_bytes(dtype);
    const StepInputs v{logits, lb * (k + 1), draft_logits, lb * k, draft, pad_in, u_accept, u_sample};
    s = check_step_disjoint(v, B, k, src, dst, in_place, tokens, n_acc, bonus, pad_out, w_new, workspace,
                            workspace_bytes, pos, mask, pm_cap, s_in, s_in_stride, s_out, s_out_stride, dev_status);
    if (s) return s;
  }
  if (B == 0) return ok();
  hipStream_t st = static_cast<hipStream_t>(stream);
  specdec::SampleLaunch sp{logits, draft_logits, dtype, draft, pad_in, u_accept, u_sample, c,
                           B, k, V, W_in, tokens, n_acc, bonus, pad_out, w_new, workspace, dev_status};
  hipError_t e = sample_launches(sp, st);
  if (e != hipSuccess) return hip_fail(e, "stochastic verify launch");
  return step_realign(k, W_in, src, dst, in_place, pad_in, tokens, n_acc, pad_out, w_new, pos, mask, pm_cap, s_in,
                      s_in_stride, s_out, s_out_stride, pad_id, dev_status, w_new_host, st);
}

specdec_status_t specdec_gather_batch(const specdec_kv_t* pool, const int32_t* pool_tok, int64_t pool_tok_stride,
                                      const int32_t* lens, const int32_t* slots, int32_t B, int32_t Lb, int32_t k,
                                      const specdec_kv_t* batch, int32_t* batch_tok, int64_t btok_stride,
                                      int32_t pad_id, int32_t* pads, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                      uint32_t* dev_status, void* stream) {
  specdec_status_t s = check_pool_pair(pool, batch, B, Lb, k, Lb, lens, slots);
  if (s) return s;
  if (B == 0) return ok();
  if (!pads) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL pads");
  if (!aligned(pads, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  if (batch_tok) {
    if (!pool_tok) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch_tok given without pool_tok");
    if (!aligned(batch_tok, 4) || !aligned(pool_tok, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "token rows not 4-byte aligned");
    if ((s = check_stride(btok_stride, static_cast<int64_t>(Lb) + 1, "btok_stride"))) return s;
    if ((s = check_stride(pool_tok_stride, 1, "pool_tok_stride"))) return s;
    if (ranges_overlap(batch_tok, static_cast<int64_t>(B) * btok_stride * 4, pool_tok,
                       static_cast<int64_t>(pool->B) * pool_tok_stride * 4))
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch and pool token rows overlap");
  }
  if ((pos == nullptr) != (mask == nullptr)) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "give both pos and mask, or neither");
  if (pos) {
    if (!aligned(pos, 8)) return fail(SPECDEC_ERR_UNSUPPORTED, "pos not 8-byte aligned");
    if (pm_cap < static_cast<int64_t>(Lb) + k + 1 || pm_cap > static_cast<int64_t>(SPECDEC_MAX_WIDTH) + SPECDEC_MAX_K + 1)
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pm_cap=%lld < Lb+k+1=%lld", (long long)pm_cap,
                  (long long)Lb + k + 1);
  }
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  {
    const int64_t b4 = 4 * static_cast<int64_t>(B), n = pos ? static_cast<int64_t>(B) * pm_cap : 0;
    s = check_disjoint({{pool->data, kv_bytes(pool), "pool"},
                        {pool_tok, batch_tok ? static_cast<int64_t>(pool->B) * pool_tok_stride * 4 : 0, "pool_tok"},
                        {lens, 4 * static_cast<int64_t>(pool->B), "lens"}, {slots, b4, "slots"}},
                       {{batch->data, kv_bytes(batch), "batch"},
                        {batch_tok, batch_tok ? static_cast<int64_t>(B) * btok_stride * 4 : 0, "batch_tok"},
                        {pads, b4, "pads"}, {pos, 8 * n, "pos"}, {mask, n, "mask"}, {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  specdec::GatherLaunch p{};
  p.pool = pool->data;
  p.pool_cap = pool->cap;
  p.N = pool->B;
  p.pool_tok = pool_tok;
  p.pool_tok_stride = pool_tok_stride;
  p.lens = lens;
  p.slots = slots;
  p.L = batch->L;
  p.B = B;
  p.H = batch->H;
  p.D = batch->D;
  p.Lb = Lb;
  p.k = k;
  p.batch = batch->data;
  p.batch_cap = batch->cap;
  p.batch_tok = batch_tok;
  p.btok_stride = btok_stride;
  p.pad_id = pad_id;
  p.pads = pads;
  p.pos = pos;
  p.mask = mask;
  p.pm_cap = pm_cap;
  p.dev_status = dev_status;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(SPECDEC_KERNEL_GATHER, st, [&] { return specdec::launch_gather(p, st); });
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  return ok();
}

specdec_status_t specdec_scatter_accepted(const specdec_kv_t* batch, const int32_t* pads, const int32_t* tokens,
                                          const int32_t* n_acc, const int32_t* slots, int32_t B, int32_t k,
                                          int32_t Lb, const specdec_kv_t* pool, int32_t* pool_tok,
                                          int64_t pool_tok_stride, int32_t* lens, int32_t* batch_tok,
                                          int64_t btok_stride, int32_t mode, uint32_t* dev_status, void* stream) {
  if (mode != SPECDEC_WRITEBACK_FULL && mode != SPECDEC_WRITEBACK_APPEND)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "write-back mode %d unknown", mode);
  specdec_status_t s = check_pool_pair(pool, batch, B, Lb, k, static_cast<int64_t>(Lb) + k + 1, lens, slots);
  if (s) return s;
  if (B == 0) return ok();
  if (!pads || !tokens || !n_acc || !pool_tok)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL pads / tokens / n_acc / pool_tok");
  if (!aligned(pads, 4) || !aligned(tokens, 4) || !aligned(n_acc, 4) || !aligned(pool_tok, 4))
    return fail(SPECDEC_ERR_UNSUPPORTED, "int32 tensor not 4-byte aligned");
  if ((s = check_stride(pool_tok_stride, 1, "pool_tok_stride"))) return s;
  if (batch_tok) {
    if (!aligned(batch_tok, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "batch_tok not 4-byte aligned");
    if ((s = check_stride(btok_stride, static_cast<int64_t>(Lb) + k + 2, "btok_stride"))) return s;
    if (ranges_overlap(batch_tok, static_cast<int64_t>(B) * btok_stride * 4, pool_tok,
                       static_cast<int64_t>(pool->B) * pool_tok_stride * 4))
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch and pool token rows overlap");
  }
  if (dev_status && !aligned(dev_status, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "dev_status not 4-byte aligned");
  {
    // the pool cache, pool token rows, lengths and batch token rows are updated
    const int64_t b4 = 4 * static_cast<int64_t>(B);
    s = check_disjoint({{batch->data, kv_bytes(batch), "batch"}, {pads, b4, "pads"},
                        {tokens, b4 * (k + 1), "tokens"}, {n_acc, b4, "n_acc"}, {slots, b4, "slots"}},
                       {{pool->data, kv_bytes(pool), "pool"},
                        {pool_tok, static_cast<int64_t>(pool->B) * pool_tok_stride * 4, "pool_tok"},
                        {lens, 4 * static_cast<int64_t>(pool->B), "lens"},
                        {batch_tok, batch_tok ? static_cast<int64_t>(B) * btok_stride * 4 : 0, "batch_tok"},
                        {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  specdec::WritebackLaunch p{};
  p.batch = batch->data;
  p.batch_cap = batch->cap;
  p.pads = pads;
  p.tokens = tokens;
  p.n_acc = n_acc;
  p.slots = slots;
  p.L = batch->L;
  p.B = B;
  p.H = batch->H;
  p.D = batch->D;
  p.k = k;
  p.Lb = Lb;
  p.pool = pool->data;
  p.pool_cap = pool->cap;
  p.N = pool->B;
  p.pool_tok = pool_tok;
  p.pool_tok_stride = pool_tok_stride;
  p.lens = lens;
  p.batch_tok = batch_tok;
  p.btok_stride = btok_stride;
  p.append_only = mode == SPECDEC_WRITEBACK_APPEND;
  p.dev_status = dev_status;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(SPECDEC_KERNEL_WRITEBACK, st, [&] { return specdec::launch_writeback(p, st); });
  if (e != hipSuccess) return hip_fail(e, "write-back launch");
  return ok();
}

specdec_status_t specdec_rollback(const int32_t* tokens, const int32_t* n_acc_in, const int32_t* pad_in, int32_t B,
                                  int32_t k, int32_t W_in, int32_t* n_acc_out, int32_t* bonus_out, int32_t* pad_out,
                                  int32_t* w_new, uint32_t* dev_status, void* stream) {
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (W_in < k + 1 || W_in > SPECDEC_MAX_WIDTH)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "W_in=%d outside [k+1=%d, %d]", W_in, k + 1, SPECDEC_MAX_WIDTH);
  if (B == 0) return ok();
  if (!tokens || !n_acc_in || !pad_in || !n_acc_out || !bonus_out || !pad_out || !w_new)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL tensor pointer");
  const void* w4[] = {tokens, n_acc_in, pad_in, n_acc_out, bonus_out, pad_out, w_new, dev_status};
  for (const void* q : w4)
    if (q && !aligned(q, 4)) return fail(SPECDEC_ERR_UNSUPPORTED, "4-byte tensor not 4-byte aligned");
  const int64_t b4 = 4 * static_cast<int64_t>(B);
  if (ranges_overlap(bonus_out, b4, n_acc_in, b4) || ranges_overlap(bonus_out, b4, pad_in, b4) ||
      ranges_overlap(bonus_out, b4, tokens, b4 * (k + 1)) || ranges_overlap(n_acc_out, b4, tokens, b4 * (k + 1)) ||
      ranges_overlap(pad_out, b4, tokens, b4 * (k + 1)) || ranges_overlap(n_acc_out, b4, pad_out, b4) ||
      ranges_overlap(bonus_out, b4, n_acc_out, b4) || ranges_overlap(bonus_out, b4, pad_out, b4) ||
      (n_acc_out != n_acc_in && ranges_overlap(n_acc_out, b4, n_acc_in, b4)) ||
      (pad_out != pad_in && ranges_overlap(pad_out, b4, pad_in, b4)) ||
      ranges_overlap(n_acc_out, b4, pad_in, b4) || ranges_overlap(pad_out, b4, n_acc_in, b4))
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "outputs overlap the inputs other than in place");
  {
    // n_acc and the paddings may be updated in place; the width and the
    // status word must stand apart from everything
    const specdec_status_t s = check_disjoint(
        {{tokens, b4 * (k + 1), "tokens"}, {n_acc_in, b4, "n_acc_in"}, {pad_in, b4, "pad_in"},
         {n_acc_out, b4, "n_acc_out"}, {bonus_out, b4, "bonus_out"}, {pad_out, b4, "pad_out"}},
        {{w_new, 4, "w_new"}, {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  specdec::RollbackLaunch p{tokens, n_acc_in, pad_in, B, k, W_in, n_acc_out, bonus_out, pad_out, w_new, dev_status};
  hipError_t e = specdec::launch_rollback(p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "rollback launch");
  return ok();
}

specdec_status_t specdec_varlen_rollback(const specdec_varlen_t* src, const specdec_varlen_t* dst,
                                         const int32_t* cu_in, const int32_t* n_acc, int32_t B, int32_t k,
                                         int32_t max_len, int32_t* cu_out, int64_t* pos, int64_t pos_cap,
                                         uint32_t* dev_status, void* stream) {
  if (!src || !dst) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL descriptor");
  if (B < 0 || B > SPECDEC_MAX_B) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "B=%d outside [0,%d]", B, SPECDEC_MAX_B);
  if (k < 0 || k > SPECDEC_MAX_K) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "k=%d outside [0,%d]", k, SPECDEC_MAX_K);
  if (src->L != dst->L || src->H != dst->H || src->D != dst->D)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "src and dst shapes differ");
  if (src->L < 0 || src->H < 1 || src->D < 1 || src->D > SPECDEC_MAX_D)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "L, H or D out of range");
  const int64_t row = static_cast<int64_t>(src->H) * src->D;
  if (row % 8 != 0) return fail(SPECDEC_ERR_UNSUPPORTED, "H*D=%lld: rows must be whole 16-byte vectors", (long long)row);
  if (src->T_cap < 0 || src->T_cap > 0x7FFFFFFFLL || dst->T_cap < src->T_cap)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "T_cap out of range or dst->T_cap < src->T_cap");
  if (max_len < k + 1) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "max_len=%d < k+1", max_len);
  if (max_len > src->T_cap) max_len = static_cast<int32_t>(src->T_cap);   // no sequence is longer
  if (B == 0) return ok();
  if (!cu_in || !n_acc || !cu_out) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL cu_in / n_acc / cu_out");
  if (!aligned(cu_in, 4) || !aligned(n_acc, 4) || !aligned(cu_out, 4) || (pos && !aligned(pos, 8)) ||
      (dev_status && !aligned(dev_status, 4)))
    return fail(SPECDEC_ERR_UNSUPPORTED, "index tensor misaligned");
  if (pos && pos_cap < src->T_cap) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "pos_cap < src T_cap");
  const int64_t bytes_src = static_cast<int64_t>(src->L) * 2 * src->T_cap * row * 2;
  const int64_t bytes_dst = static_cast<int64_t>(dst->L) * 2 * dst->T_cap * row * 2;
  if (src->L > 0 && src->T_cap > 0) {
    if (!src->data || !dst->data) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL cache data");
    if (!aligned(src->data, 16) || !aligned(dst->data, 16)) return fail(SPECDEC_ERR_UNSUPPORTED, "cache not 16-byte aligned");
    if (ranges_overlap(src->data, bytes_src, dst->data, bytes_dst))
      return fail(SPECDEC_ERR_INVALID_ARGUMENT, "src and dst caches overlap");
  }
  const int64_t c4 = 4 * (static_cast<int64_t>(B) + 1);
  {
    const bool data = src->L > 0 && src->T_cap > 0;
    specdec_status_t s = check_disjoint(
        {{cu_in, c4, "cu_in"}, {n_acc, 4 * static_cast<int64_t>(B), "n_acc"}, {data ? src->data : nullptr, bytes_src, "src"}},
        {{cu_out, c4, "cu_out"}, {pos, pos ? 8 * pos_cap : 0, "pos"}, {data ? dst->data : nullptr, bytes_dst, "dst"},
         {dev_status, 4, "dev_status"}});
    if (s) return s;
  }
  if (static_cast<int64_t>(src->L) * 2 * B > 0xFFFFFFFFLL) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "too many spans");
  specdec::VarlenLaunch p{src->data, dst->data, src->T_cap, dst->T_cap, src->L, src->H, src->D, cu_in, n_acc,
                          B, k, max_len, cu_out, pos, dev_status};
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = timed(SPECDEC_KERNEL_VARLEN, st, [&] { return specdec::launch_varlen_rollback(p, st); });
  if (e != hipSuccess) return hip_fail(e, "variable-length rollback launch");
  return ok();
}

specdec_status_t specdec_timing_enable(int32_t kernel_mask) {
  if (kernel_mask < 0 || kernel_mask > SPECDEC_TIMING_ALL)
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "timing mask %d outside [0,%d]", kernel_mask, SPECDEC_TIMING_ALL);
  Timers& t = timers();
  std::lock_guard<std::mutex> lk(t.mu);
  t.mask = kernel_mask;
  return ok();
}

specdec_status_t specdec_timing_reset(void) {
  Timers& t = timers();
  std::lock_guard<std::mutex> lk(t.mu);
  try {
    t.pool.reserve(t.pool.size() + 2 * t.pending.size());   // the pushes below do not allocate
  } catch (...) {
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "out of host memory");
  }
  for (const TimedLaunch& p : t.pending) {
    (void)hipEventSynchronize(p.end);
    t.pool.push_back(p.begin);
    t.pool.push_back(p.end);
  }
  t.pending.clear();
  for (int i = 0; i < kTimedKernels; ++i) {
    t.total_ms[i] = 0;
    t.launches[i] = 0;
  }
  return ok();
}

specdec_status_t specdec_timing_query(int32_t kernel, double* total_ms, int64_t* launches) {
  if (kernel < 0 || kernel >= kTimedKernels) return fail(SPECDEC_ERR_INVALID_ARGUMENT, "unknown kernel id %d", kernel);
  Timers& t = timers();
  std::lock_guard<std::mutex> lk(t.mu);
  try {
    t.pool.reserve(t.pool.size() + 2 * t.pending.size());   // the pushes below do not allocate
  } catch (...) {
    return fail(SPECDEC_ERR_INVALID_ARGUMENT, "out of host memory");
  }
  size_t done = 0;
  for (; done < t.pending.size(); ++done) {
    const TimedLaunch& p = t.pending[done];
    hipError_t e = hipEventSynchronize(p.end);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.begin, p.end);
    if (e != hipSuccess) {
      // launches already added are dropped from the queue; the failing one stays
      t.pending.erase(t.pending.begin(), t.pending.begin() + static_cast<std::ptrdiff_t>(done));
      return hip_fail(e, "timer event");
    }
    t.total_ms[p.kernel] += ms;
    t.launches[p.kernel] += 1;
    t.pool.push_back(p.begin);
    t.pool.push_back(p.end);
  }
  t.pending.clear();
  if (total_ms) *total_ms = t.total_ms[kernel];
  if (launches) *launches = t.launches[kernel];
  return ok();
}

}  // extern "C"
