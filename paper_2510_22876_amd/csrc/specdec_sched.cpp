// The SequencePool scheduler of EXSpec (arXiv 2510.22876, Algorithm 2;
// Section 3.2, "Cross-Batch Scheduling"): host-side bookkeeping of a pool of
// ragged sequences and the choice of each step's batch over a sliding window
// (lazy realignment, same-length grouping, unpad-repad fallback).  No GPU
// call is made here; the batch it picks is moved by specdec_gather_batch and
// written back by specdec_scatter_accepted.
#include <algorithm>
#include <map>
#include <new>
#include <vector>

#include "specdec.h"
#include "specdec_internal.h"

struct specdec_sched {
  int32_t N = 0, window = 0, batch = 0, max_new = 0, eos_id = -1;
  std::vector<int32_t> active_order;  // active sequences in pool order
  std::vector<int32_t> len, generated;
  std::vector<uint8_t> active;
  std::vector<int32_t> prev;          // previous batch, kept while it stays rectangular
  bool has_prev = false;
  // the batch handed out by next_batch and not yet committed
  std::vector<int32_t> cur;
  specdec_batch_info_t cur_info{};
  bool has_cur = false;
};

namespace {

specdec_status_t sched_fail(specdec_status_t code, const char* msg) {
  specdec::set_last_error(msg);
  return code;
}

specdec_status_t sched_ok() {
  specdec::clear_last_error();
  return SPECDEC_OK;
}

void choose(specdec_sched* s) {
  specdec_batch_info_t info{};
  s->cur.clear();
  // the window: the first `window` active sequences in pool order
  const size_t wn = std::min(static_cast<size_t>(s->window), s->active_order.size());
  if (wn == 0) {
    s->cur_info = info;
    return;
  }
  bool prev_alive = s->has_prev;
  if (prev_alive)
    for (int32_t q : s->prev) prev_alive = prev_alive && s->active[q];
  bool reuse = false;
  if (prev_alive) {
    // lazy realignment: every row accepted alike, the batch is still rectangular
    s->cur = s->prev;
    reuse = true;
  } else {
    const int32_t b = static_cast<int32_t>(std::min(static_cast<size_t>(s->batch), wn));
    std::map<int32_t, std::vector<int32_t>> buckets;  // length -> members in pool order
    for (size_t j = 0; j < wn; ++j) {
      const int32_t q = s->active_order[j];
      buckets[s->len[q]].push_back(q);
    }
    const std::vector<int32_t>& first = buckets[s->len[s->active_order[0]]];
    const std::vector<int32_t>* pick = nullptr;
    if (static_cast<int32_t>(first.size()) >= b) {
      pick = &first;
    } else {
      // the largest bucket with at least b members; among equal sizes the
      // shorter length (the map is in increasing length order)
      for (const auto& kvp : buckets)
        if (static_cast<int32_t>(kvp.second.size()) >= b && (!pick || kvp.second.size() > pick->size()))
          pick = &kvp.second;
    }
    if (pick) s->cur.assign(pick->begin(), pick->begin() + b);
    else s->cur.assign(s->active_order.begin(), s->active_order.begin() + b);
  }
  int32_t lo = s->len[s->cur[0]], hi = lo;
  for (int32_t q : s->cur) {
    lo = std::min(lo, s->len[q]);
    hi = std::max(hi, s->len[q]);
  }
  info.B = static_cast<int32_t>(s->cur.size());
  info.width = hi;
  info.same_length = lo == hi ? 1 : 0;
  info.reuse = reuse ? 1 : 0;
  s->cur_info = info;
}

// Runs a body that may allocate; no exception crosses the C ABI.
template <typename F>
specdec_status_t guarded(F&& body) {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "out of host memory");
  } catch (...) {
    return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "unexpected host error");
  }
}

}  // namespace

extern "C" {

specdec_status_t specdec_sched_create(const int32_t* lens, int32_t N, int32_t window, int32_t batch,
                                      int32_t max_new, int32_t sort_by_length, int32_t eos_id,
                                      specdec_sched_t** out) {
  if (!out) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  if (N < 0 || N > (1 << 26)) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "N outside [0, 2^26]");
  if (N > 0 && !lens) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "lens is NULL");
  if (window < 1 || batch < 1) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "window and batch must be positive");
  if (batch > SPECDEC_MAX_B) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "batch above SPECDEC_MAX_B");
  if (max_new < 1) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "max_new must be positive");
  for (int32_t i = 0; i < N; ++i)
    if (lens[i] < 0 || lens[i] > SPECDEC_MAX_WIDTH)
      return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "a length is outside [0, SPECDEC_MAX_WIDTH]");
  return guarded([&] {
    specdec_sched* s = new specdec_sched;
    try {
      s->N = N;
      s->window = window;
      s->batch = batch;
      s->max_new = max_new;
      s->eos_id = eos_id;
      s->len.assign(lens, lens + N);
      s->generated.assign(N, 0);
      s->active.assign(N, 1);
      s->active_order.resize(N);
      for (int32_t i = 0; i < N; ++i) s->active_order[i] = i;
      if (sort_by_length)
        std::stable_sort(s->active_order.begin(), s->active_order.end(),
                         [s](int32_t a, int32_t b) { return s->len[a] < s->len[b]; });
    } catch (...) {
      delete s;
      throw;
    }
    *out = s;
    return sched_ok();
  });
}

void specdec_sched_destroy(specdec_sched_t* s) { delete s; }

specdec_status_t specdec_sched_next_batch(specdec_sched_t* s, int32_t* slots, int32_t* lens,
                                          specdec_batch_info_t* info) {
  if (!s || !slots || !info) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL scheduler / slots / info");
  if (!s->has_cur) {
    const specdec_status_t st = guarded([&] {
      choose(s);
      return SPECDEC_OK;
    });
    if (st) return st;
    s->has_cur = s->cur_info.B > 0;
  }
  *info = s->cur_info;
  for (int32_t i = 0; i < s->cur_info.B; ++i) {
    slots[i] = s->cur[i];
    if (lens) lens[i] = s->len[s->cur[i]];
  }
  return sched_ok();
}

specdec_status_t specdec_sched_commit(specdec_sched_t* s, const int32_t* n_acc, const int32_t* tokens, int32_t k) {
  if (!s || !n_acc) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL scheduler / n_acc");
  if (!s->has_cur) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "no batch to commit (call next_batch first)");
  if (k < 0 || k > SPECDEC_MAX_K) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "k outside [0, SPECDEC_MAX_K]");
  if (s->eos_id >= 0 && !tokens) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "tokens are needed to detect eos");
  const int32_t B = s->cur_info.B;
  for (int32_t i = 0; i < B; ++i) {
    if (n_acc[i] < 0 || n_acc[i] > k) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "n_acc outside [0, k]");
    if (static_cast<int64_t>(s->len[s->cur[i]]) + n_acc[i] + 1 > SPECDEC_MAX_WIDTH)
      return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "a sequence would exceed SPECDEC_MAX_WIDTH");
  }
  bool uniform = true, deactivated = false;
  for (int32_t i = 0; i < B; ++i) {
    const int32_t q = s->cur[i];
    const int32_t a = n_acc[i] + 1;
    s->len[q] += a;
    s->generated[q] += a;
    bool done = s->generated[q] >= s->max_new;
    if (s->eos_id >= 0)
      for (int32_t r = 0; r < a && !done; ++r) done = tokens[static_cast<int64_t>(i) * (k + 1) + r] == s->eos_id;
    if (done) {
      s->active[q] = 0;
      deactivated = true;
    }
    uniform = uniform && n_acc[i] == n_acc[0];
  }
  if (deactivated)
    s->active_order.erase(std::remove_if(s->active_order.begin(), s->active_order.end(),
                                         [s](int32_t q) { return !s->active[q]; }),
                          s->active_order.end());
  s->has_prev = uniform;
  if (uniform) {
    const specdec_status_t st = guarded([&] {
      s->prev = s->cur;
      return SPECDEC_OK;
    });
    if (st) {
      s->has_prev = false;
      s->has_cur = false;
      return st;
    }
  }
  s->has_cur = false;
  return sched_ok();
}

specdec_status_t specdec_sched_lengths(const specdec_sched_t* s, int32_t* lens) {
  if (!s || (!lens && s->N > 0)) return sched_fail(SPECDEC_ERR_INVALID_ARGUMENT, "NULL scheduler / lens");
  std::copy(s->len.begin(), s->len.end(), lens);
  return sched_ok();
}

int32_t specdec_sched_active(const specdec_sched_t* s) {
  return s ? static_cast<int32_t>(s->active_order.size()) : 0;
}

}  // extern "C"
