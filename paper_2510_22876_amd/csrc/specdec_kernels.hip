// HIP kernels for one greedy verify + KV realign step (EqSpec, arXiv 2510.22876)
// on MI355X (gfx950, wave64).
//
//   verify_partial     vocab-wide argmax of every logit row (Algorithm 3), split
//                      over workgroups per row; each workgroup stores its
//                      packed (key, index) maximum in its own workspace slot.
//   verify_finalize    one workgroup: reduces the slots of each row, then the
//                      prefix-match scan, the bonus token and the new width /
//                      paddings (Eq. (1), Eq. (2)).  Two launches instead of a
//                      last-workgroup-done counter: a device-scope fence and
//                      atomic per workgroup costs more than a kernel boundary.
//   realign_oop        out-of-place unpad-append-repad of the bf16 KV cache:
//                      one workgroup per 16 KB chunk of a (layer, K/V, row,
//                      head) span, 128-bit loads and stores.
//   realign_inplace    in-place variant: one workgroup walks a whole span in
//                      the direction of its shift, a barrier between the reads
//                      and the writes of each chunk.
//   posmask blocks     position ids / mask of invariant I2, appended to either
//                      realign grid (or launched alone).
//
// Everything here is bandwidth-bound data movement plus integer compares: no
// matrix cores.
#include <cstdlib>

#include "posmask.h"
#include "span_copy.h"
#include "specdec_internal.h"

namespace specdec {
namespace {

constexpr uint32_t kBadPadIn = 0x1u, kBadAccept = 0x2u, kBadWidth = 0x4u, kBadPadOut = 0x8u;
constexpr int kWaves = kThreads / 64;
constexpr int kPmColsPerBlock = 4 * kThreads;

// ---------------------------------------------------------------------------
// argmax keys
//
// A logit is mapped to an unsigned key whose integer order is the order of
// the values: -0.0 and +0.0 share a key, every NaN gets the largest key (a NaN
// ranks above every number).  Within a thread elements are visited in
// increasing index order and only a strictly larger key replaces the best,
// so the lowest index wins among equal keys; across threads the pair is
// packed as (key << 32) | ~index, whose maximum again prefers the lowest
// index.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t key_f32(uint32_t u) {
  const uint32_t mag = u & 0x7FFFFFFFu;
  if (mag > 0x7F800000u) return 0xFFFFFFFFu;
  if (mag == 0u) return 0x80000000u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// 16-bit logits: a positive h maps to h | 0x8000, a negative one to
// (h ^ 0xFFFF) + 1 (so -0.0 lands on +0.0's key 0x8000), a NaN to 0xFFFF.
template <uint32_t kNanMag>  // 0x7F80 for bf16, 0x7C00 for f16
__device__ __forceinline__ uint32_t key_16(uint32_t h) {
  if ((h & 0x7FFFu) > kNanMag) return 0xFFFFu;
  return (h & 0x8000u) ? ((h ^ 0xFFFFu) + 1u) : (h | 0x8000u);
}

typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// The keys of both halves of a word with packed 16-bit operations, exact
// except for NaNs (which land outside the keys of -inf..+inf).
__device__ __forceinline__ u16x2 keys2(uint32_t w) {
  const s16x2 sign = __builtin_bit_cast(s16x2, w) >> (s16x2){15, 15};   // 0xFFFF on negative halves
  const uint32_t m = __builtin_bit_cast(uint32_t, sign);
  return __builtin_bit_cast(u16x2, w ^ (m | 0x80008000u)) + __builtin_bit_cast(u16x2, m & 0x00010001u);
}

struct Best {
  uint32_t key = 0u;
  int32_t idx = 0;
  __device__ __forceinline__ void take(uint32_t k, int32_t i) {
    if (k > key) {
      key = k;
      idx = i;
    }
  }
};

template <int DT>
struct Logit;

template <>
struct Logit<0> {  // f32
  static constexpr int kBytes = 4;
  __device__ static uint32_t key_at(const char* row, int64_t i) {
    return key_f32(*reinterpret_cast<const uint32_t*>(row + 4 * i));
  }
  __device__ static void take_vec(Best& b, const uint4& q, int32_t e) {
    b.take(key_f32(q.x), e);
    b.take(key_f32(q.y), e + 1);
    b.take(key_f32(q.z), e + 2);
    b.take(key_f32(q.w), e + 3);
  }
};

template <uint32_t kNanMag>
struct Logit16 {
  static constexpr int kBytes = 2;
  __device__ static uint32_t key_at(const char* row, int64_t i) {
    return key_16<kNanMag>(*reinterpret_cast<const uint16_t*>(row + 2 * i));
  }
  static constexpr uint32_t kPosInf = kNanMag | 0x8000u;                  // key of +inf
  static constexpr uint32_t kNegInf = ((kNanMag | 0x8000u) ^ 0xFFFFu) + 1u;  // key of -inf
  // Largest key of a 16-byte vector of 8 logits (0xFFFF if it holds a NaN).
  __device__ static uint32_t vec_key(const uint4& q) {
    const u16x2 a = keys2(q.x), b = keys2(q.y), c = keys2(q.z), d = keys2(q.w);
    const u16x2 hi = __builtin_elementwise_max(__builtin_elementwise_max(a, b), __builtin_elementwise_max(c, d));
    const u16x2 lo = __builtin_elementwise_min(__builtin_elementwise_min(a, b), __builtin_elementwise_min(c, d));
    const uint32_t vmax = hi.x > hi.y ? hi.x : hi.y;
    const uint32_t vmin = lo.x < lo.y ? lo.x : lo.y;
    return (vmax > kPosInf || vmin < kNegInf) ? 0xFFFFu : vmax;
  }
  // The lowest element of vector q (first element index e) whose key is k.
  __device__ static void take_in_vec(Best& b, const uint4& q, uint32_t k, int32_t e) {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    int32_t at = e + 7;
#pragma unroll
    for (int j = 7; j >= 0; --j) {
      const uint32_t h = (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
      if (key_16<kNanMag>(h) == k) at = e + j;
    }
    b.take(k, at);
  }
};
template <>
struct Logit<1> : Logit16<0x7F80u> {};  // bf16
template <>
struct Logit<2> : Logit16<0x7C00u> {};  // f16

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

__device__ __forceinline__ int32_t wave_max_i32(int32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

struct VerifyArgs {
  const char* logits;
  const int32_t* draft;
  const int32_t* pad_in;
  int32_t B, k, V, W_in;
  int32_t* tokens;
  int32_t* n_acc;
  int32_t* bonus;
  int32_t* pad_out;
  int32_t* w_new;
  unsigned long long* partial;  // [B*(k+1)][chunks] packed maxima
  uint32_t* dev_status;
  int64_t chunk_elems;
  int32_t chunks;               // workgroups per logit row
  int32_t* order;               // in-place realignment order table (NULL: not written)
};

// Tunables of the vocabulary scan (compile-time; chosen by sweeping on
// MI355X with the logits read from HBM):
//   SPECDEC_VERIFY_UNROLL     16-byte loads per thread in flight per iteration
//   SPECDEC_VERIFY_TARGET     workgroups the scan aims for in total
//   SPECDEC_VERIFY_MIN_CHUNK / SPECDEC_VERIFY_MAX_CHUNK  logits per workgroup
#ifndef SPECDEC_VERIFY_UNROLL
#define SPECDEC_VERIFY_UNROLL 4
#endif
#ifndef SPECDEC_VERIFY_TARGET
#define SPECDEC_VERIFY_TARGET 2048
#endif
#ifndef SPECDEC_VERIFY_MIN_CHUNK
#define SPECDEC_VERIFY_MIN_CHUNK 2048
#endif
#ifndef SPECDEC_VERIFY_MAX_CHUNK
#define SPECDEC_VERIFY_MAX_CHUNK 16384
#endif
// In-place realignment order that the merge writes: length classes of the
// moving rows (longest first; 1: every moving row in the cache's order), and
// rows per group of the walk (the walk takes the rows a group at a time, each
// group slab by slab in the cache's order)
#ifndef SPECDEC_INPLACE_CLASSES
#define SPECDEC_INPLACE_CLASSES 2
#endif
#ifndef SPECDEC_INPLACE_ROWGROUP
#define SPECDEC_INPLACE_ROWGROUP 32
#endif

// Scan logit elements [beg, end) of one row; 16-byte vectors over the aligned
// interior, single elements for the unaligned head and the tail.
template <int DT, int kTpb = kThreads, int kUnroll = SPECDEC_VERIFY_UNROLL>
__device__ __forceinline__ void scan_range(const char* row, int64_t beg, int64_t end, Best& b) {
  using T = Logit<DT>;
  constexpr int kPerVec = 16 / T::kBytes;
  const int tid = threadIdx.x;
  const uintptr_t addr = reinterpret_cast<uintptr_t>(row) + static_cast<uintptr_t>(beg) * T::kBytes;
  int64_t head = static_cast<int64_t>((16u - (addr & 15u)) & 15u) / T::kBytes;
  if (head > end - beg) head = end - beg;
  const int64_t a0 = beg + head;
  const int64_t nvec = (end - a0) / kPerVec;
  const int64_t a1 = a0 + nvec * kPerVec;
  if (tid < head) b.take(T::key_at(row, beg + tid), static_cast<int32_t>(beg + tid));
  const uint4* vp = reinterpret_cast<const uint4*>(row + a0 * T::kBytes);
  if constexpr (T::kBytes == 2) {
    // per vector only its largest key; the first vector (lowest index) holding
    // this thread's largest key is kept in registers and searched at the end
    uint32_t vk = 0u;
    int32_t ve = -1;
    uint4 vq = make_uint4(0u, 0u, 0u, 0u);
    for (int64_t v0 = 0; v0 < nvec; v0 += kTpb * kUnroll) {
      uint4 q[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t v = v0 + u * kTpb + tid;
        q[u] = v < nvec ? vp[v] : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t v = v0 + u * kTpb + tid;
        const uint32_t k = T::vec_key(q[u]);
        if (v < nvec && k > vk) {
          vk = k;
          ve = static_cast<int32_t>(a0 + v * kPerVec);
          vq = q[u];
        }
      }
    }
    if (ve >= 0) T::take_in_vec(b, vq, vk, ve);
  } else {
    for (int64_t v0 = 0; v0 < nvec; v0 += kTpb * kUnroll) {
      uint4 q[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t v = v0 + u * kTpb + tid;
        q[u] = v < nvec ? vp[v] : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int64_t v = v0 + u * kTpb + tid;
        if (v < nvec) T::take_vec(b, q[u], static_cast<int32_t>(a0 + v * kPerVec));
      }
    }
  }
  if (tid < end - a1) b.take(T::key_at(row, a1 + tid), static_cast<int32_t>(a1 + tid));
}

template <int DT>
__global__ __launch_bounds__(kThreads) void verify_partial_kernel(VerifyArgs a) {
  __shared__ unsigned long long wkey[kWaves];
  const int64_t row = blockIdx.x / a.chunks;
  const int64_t chunk = blockIdx.x - row * a.chunks;
  const int64_t beg = chunk * a.chunk_elems;
  int64_t end = beg + a.chunk_elems;
  if (end > a.V) end = a.V;
  const char* rowp = a.logits + row * static_cast<int64_t>(a.V) * Logit<DT>::kBytes;

  Best b;
  scan_range<DT>(rowp, beg, end, b);
  unsigned long long key =
      (static_cast<unsigned long long>(b.key) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(b.idx));
  key = wave_max_u64(key);
  if ((threadIdx.x & 63) == 0) wkey[threadIdx.x >> 6] = key;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long k2 = wkey[0];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) k2 = wkey[q] > k2 ? wkey[q] : k2;
    a.partial[blockIdx.x] = k2;
  }
}

constexpr int kFinalizeThreads = 1024;
constexpr int kInClasses = SPECDEC_INPLACE_CLASSES;
constexpr uint32_t kInRowGroup = SPECDEC_INPLACE_ROWGROUP;

// Geometry of row i after verification: ok (pad_in in range), the new length
// and padding; the row moves when its padding changes.
struct RowMove {
  bool ok, moves;
  int32_t p, po, len;
};
__device__ __forceinline__ RowMove row_move(const VerifyArgs& a, int i, int32_t w) {
  const int32_t L = a.W_in - (a.k + 1);
  RowMove m;
  m.p = a.pad_in[i];
  m.ok = m.p >= 0 && m.p <= L;
  m.len = (L - m.p) + a.n_acc[i] + 1;
  m.po = w - m.len;
  m.moves = m.ok && m.po != m.p;
  return m;
}

// The in-place realignment order (one workgroup of kFinalizeThreads, after
// the paddings): moving rows in kInClasses classes of equal length range,
// longest first, then the rows with nothing to move; each class in
// increasing row order (a stable partition: per chunk of rows a ballot per
// class, then prefixes over the waves).  The in-place walk takes the spans
// of the longest rows first, so that the longest walks do not start last.
__device__ void write_inplace_order(const VerifyArgs& a, int32_t w) {
  constexpr int kW = kFinalizeThreads / 64;
  constexpr int kCls = kInClasses + 1;   // the last class: rows with nothing to move
  __shared__ int32_t s_lo[kW], s_hi[kW];
  __shared__ int32_t s_cnt[kCls], s_start[kCls], s_carry[kCls];
  __shared__ int32_t s_wave[kCls][kW];
  static_assert(kInClasses >= 1 && kCls <= kMaxOrderClasses, "order classes");
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int32_t lo = 0x7FFFFFFF, hi = 0;
  for (int i = tid; i < a.B; i += kFinalizeThreads) {
    const RowMove m = row_move(a, i, w);
    if (m.moves) {
      lo = m.len < lo ? m.len : lo;
      hi = m.len > hi ? m.len : hi;
    }
  }
  hi = wave_max_i32(hi);
  lo = -wave_max_i32(-lo);
  if (lane == 0) {
    s_hi[wv] = hi;
    s_lo[wv] = lo;
  }
  if (tid < kCls) {
    s_cnt[tid] = 0;
    s_carry[tid] = 0;
  }
  __syncthreads();
  hi = s_hi[0];
  lo = s_lo[0];
#pragma unroll
  for (int q = 1; q < kW; ++q) {
    hi = s_hi[q] > hi ? s_hi[q] : hi;
    lo = s_lo[q] < lo ? s_lo[q] : lo;
  }
  const int64_t range = static_cast<int64_t>(hi) - lo + 1;
  auto cls = [&](const RowMove& m) {
    if (!m.moves) return kInClasses;
    const int64_t c = (static_cast<int64_t>(hi) - m.len) * kInClasses / range;
    return static_cast<int>(c < kInClasses ? c : kInClasses - 1);
  };
  for (int i = tid; i < a.B; i += kFinalizeThreads) atomicAdd(&s_cnt[cls(row_move(a, i, w))], 1);
  __syncthreads();
  if (tid == 0) {
    int32_t acc = 0;
    for (int c = 0; c < kCls; ++c) {
      s_start[c] = acc;
      acc += s_cnt[c];
    }
  }
  __syncthreads();
  for (int base = 0; base < a.B; base += kFinalizeThreads) {
    const int i = base + tid;
    RowMove m{};
    int c = kCls;   // past the end of the batch
    if (i < a.B) {
      m = row_move(a, i, w);
      c = cls(m);
    }
    int rank = 0;
#pragma unroll
    for (int cc = 0; cc < kCls; ++cc) {
      const unsigned long long bits = __ballot(c == cc);
      if (lane == 0) s_wave[cc][wv] = __popcll(bits);
      if (c == cc) rank = __popcll(bits & ((1ull << lane) - 1ull));
    }
    __syncthreads();
    if (c < kCls) {
      int32_t pos = s_start[c] + s_carry[c] + rank;
      for (int q = 0; q < wv; ++q) pos += s_wave[c][q];
      int32_t* e = a.order + 4 * static_cast<int64_t>(pos);   // four words (the workspace is 8-byte aligned)
      e[0] = i;
      e[1] = m.p;
      e[2] = m.moves ? m.po : m.p;   // nothing to move: equal paddings
      e[3] = m.len;
    }
    __syncthreads();
    if (tid < kCls) {
      int32_t add = 0;
      for (int q = 0; q < kW; ++q) add += s_wave[tid][q];
      s_carry[tid] += add;
    }
    __syncthreads();
  }
}

// One workgroup of kFinalizeThreads: row maxima, then per sequence the
// prefix-match scan, the bonus token and its new length; then the width and
// the paddings.

__global__ __launch_bounds__(kFinalizeThreads) void verify_finalize_kernel(VerifyArgs a) {
  __shared__ int32_t wmax[kFinalizeThreads / 64];
  const int32_t L = a.W_in - (a.k + 1);
  const int kp1 = a.k + 1;
  const int64_t rows = static_cast<int64_t>(a.B) * kp1;
  // row maxima -> predicted tokens
  for (int64_t r = threadIdx.x; r < rows; r += kFinalizeThreads) {
    const unsigned long long* p = a.partial + r * a.chunks;
    unsigned long long m = p[0];
    for (int c = 1; c < a.chunks; ++c) m = p[c] > m ? p[c] : m;
    a.tokens[r] = static_cast<int32_t>(~static_cast<uint32_t>(m & 0xFFFFFFFFull));
  }
  __syncthreads();  // tokens written by this workgroup are visible to it
  int32_t local = 0;
  for (int i = threadIdx.x; i < a.B; i += kFinalizeThreads) {
    const int32_t p = a.pad_in[i];
    const bool ok = p >= 0 && p <= L;
    const int32_t* tok = a.tokens + static_cast<int64_t>(i) * kp1;
    const int32_t* dr = a.draft + static_cast<int64_t>(i) * a.k;
    int32_t nacc = a.k;
    for (int r = 0; r < a.k; ++r)
      if (dr[r] != tok[r]) {
        nacc = r;
        break;
      }
    a.n_acc[i] = nacc;
    if (a.bonus) a.bonus[i] = tok[nacc];
    if (ok) {
      const int32_t len = (L - p) + nacc + 1;
      local = len > local ? len : local;
    } else if (a.dev_status) {
      atomicOr(a.dev_status, kBadPadIn);
    }
  }
  local = wave_max_i32(local);
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = local;
  __syncthreads();
  int32_t w = wmax[0];
#pragma unroll
  for (int q = 1; q < kFinalizeThreads / 64; ++q) w = wmax[q] > w ? wmax[q] : w;
  for (int i = threadIdx.x; i < a.B; i += kFinalizeThreads) {
    const int32_t p = a.pad_in[i];
    const bool ok = p >= 0 && p <= L;
    a.pad_out[i] = ok ? w - ((L - p) + a.n_acc[i] + 1) : -1;
  }
  if (threadIdx.x == 0) a.w_new[0] = w;
  if (a.order) write_inplace_order(a, w);
}

// One launch of greedy verification for batches whose logit rows are short
// enough for one workgroup each (used where the library owns the scratch and
// so knows its counters start at zero).  Every workgroup scans one whole row
// and writes its prediction; the last row of a sequence to finish (an
// agent-scope acquire-release count per sequence) does that sequence's
// prefix-match scan, bonus token and new length; the last sequence to finish
// (one more count) computes the width and the paddings.  A release fence
// costs a serialized L2 write-back on this GPU (about 19 ns each, measured),
// so the design keeps one count per row and one per sequence, never one per
// chunk of a row.  No workgroup waits for another: each one counts and either
// exits or, being last, carries on.
struct FusedVerifyArgs {
  VerifyArgs v;
  uint32_t* seq_count;    // [B], zero on entry
  uint32_t* batch_count;  // [1], zero on entry
  int32_t* lens;          // [B] new lengths (0 for a row with a bad pad_in)
};

constexpr int kFusedThreads = 1024, kFusedUnroll = 8, kFusedWaves = kFusedThreads / 64;
static_assert(kFusedThreads * kFusedUnroll * 16 >= 128 * 1024, "a fused row is one iteration of loads");

template <int DT>
__global__ __launch_bounds__(kFusedThreads) void verify_fused_kernel(FusedVerifyArgs f) {
  const VerifyArgs& a = f.v;
  __shared__ unsigned long long wkey[kFusedWaves];
  __shared__ int32_t wmax[kFusedWaves];
  __shared__ int seq_last, batch_last;   // one flag per stage: no wave reads a flag another stage rewrites
  const int64_t row = blockIdx.x;
  const int kp1 = a.k + 1;
  const int i = static_cast<int>(row / kp1);
  Best b;
  scan_range<DT, kFusedThreads, kFusedUnroll>(a.logits + row * static_cast<int64_t>(a.V) * Logit<DT>::kBytes, 0,
                                              a.V, b);
  unsigned long long key =
      (static_cast<unsigned long long>(b.key) << 32) | static_cast<uint32_t>(~static_cast<uint32_t>(b.idx));
  key = wave_max_u64(key);
  if ((threadIdx.x & 63) == 0) wkey[threadIdx.x >> 6] = key;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long k2 = wkey[0];
#pragma unroll
    for (int q = 1; q < kFusedWaves; ++q) k2 = wkey[q] > k2 ? wkey[q] : k2;
    a.tokens[row] = static_cast<int32_t>(~static_cast<uint32_t>(k2 & 0xFFFFFFFFull));
    const uint32_t before = __hip_atomic_fetch_add(f.seq_count + i, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    seq_last = before == static_cast<uint32_t>(a.k);
  }
  __syncthreads();
  if (!seq_last) return;
  // the sequence's k+1 predictions are all written: wave 0 makes them visible
  // to itself and loads them, and the drafts, at once (one lane per slot)
  if (threadIdx.x < 64) {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int lane = static_cast<int>(threadIdx.x);
    const int32_t L = a.W_in - kp1;
    const int32_t* tok = a.tokens + static_cast<int64_t>(i) * kp1;
    const int32_t* dr = a.draft + static_cast<int64_t>(i) * a.k;
    const int32_t t = lane <= a.k ? tok[lane] : 0;
    const int32_t d = lane < a.k ? dr[lane] : 0;
    const int32_t t_last = tok[a.k];                       // the prediction after the last draft (lane 64 for k = 64)
    const unsigned long long miss = __ballot(lane < a.k && d != t);
    const int32_t nacc = miss ? static_cast<int32_t>(__builtin_ctzll(miss)) : a.k;
    const int32_t bon = __shfl(t, nacc < 64 ? nacc : 0);
    if (lane == 0) {
      const int32_t p = a.pad_in[i];
      a.n_acc[i] = nacc;
      if (a.bonus) a.bonus[i] = nacc < 64 ? bon : t_last;
      const bool ok = p >= 0 && p <= L;
      f.lens[i] = ok ? (L - p) + nacc + 1 : 0;           // 0: left out of the width, padding -1
      if (!ok && a.dev_status) atomicOr(a.dev_status, kBadPadIn);
      const uint32_t before = __hip_atomic_fetch_add(f.batch_count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      batch_last = before == static_cast<uint32_t>(a.B - 1);
    }
  }
  __syncthreads();
  if (!batch_last) return;
  // every sequence's length is written; each wave makes them visible to
  // itself, and one load of each length gives both the width and the padding
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  constexpr int kPer = kMaxFusedVerifyRows / kFusedThreads;   // sequences per thread at most (B <= rows)
  int32_t len[kPer];
  int32_t local = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int q = static_cast<int>(threadIdx.x) + j * kFusedThreads;
    len[j] = q < a.B ? f.lens[q] : 0;
    local = len[j] > local ? len[j] : local;
  }
  local = wave_max_i32(local);
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = local;
  __syncthreads();
  int32_t w = wmax[0];
#pragma unroll
  for (int q = 1; q < kFusedWaves; ++q) w = wmax[q] > w ? wmax[q] : w;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int q = static_cast<int>(threadIdx.x) + j * kFusedThreads;
    if (q < a.B) a.pad_out[q] = len[j] > 0 ? w - len[j] : -1;
  }
  if (threadIdx.x == 0) a.w_new[0] = w;
}

// ---------------------------------------------------------------------------
// realign
//
// Tunables (compile-time; the defaults were chosen by sweeping on MI355X):
//   *_VEC  16-byte vectors per lane per chunk (out of place: pieces per
//          workgroup)
//   *_TPB  threads per workgroup (a multiple of 64)
//   OOP_SPLIT  distance in vectors between the pieces of an out-of-place
//          workgroup
//   *_NT   nontemporal hints (the cache is streamed once): bit 0 on loads,
//          bit 1 on stores
// Small, in-order workgroups keep the set of DRAM rows touched at any moment
// compact; spreading a workgroup's pieces apart keeps that pattern while
// halving the number of workgroups, which matters where a workgroup only
// stores (padding) and the dispatch rate would otherwise bound the kernel.
// ---------------------------------------------------------------------------
#ifndef SPECDEC_OOP_VEC
#define SPECDEC_OOP_VEC 2
#endif
#ifndef SPECDEC_OOP_TPB
#define SPECDEC_OOP_TPB 64
#endif
#ifndef SPECDEC_OOP_SPLIT
#define SPECDEC_OOP_SPLIT 512
#endif
#ifndef SPECDEC_OOP_NT
#define SPECDEC_OOP_NT 3
#endif
#ifndef SPECDEC_INPLACE_VEC
#define SPECDEC_INPLACE_VEC 32
#endif
#ifndef SPECDEC_INPLACE_TPB
#define SPECDEC_INPLACE_TPB 256
#endif
#ifndef SPECDEC_INPLACE_NT
#define SPECDEC_INPLACE_NT 3
#endif

struct RealignArgs {
  const u32x4* src;
  u32x4* dst;
  int64_t src_span_vecs, dst_span_vecs;  // cap * D / 8
  int32_t vpc;                           // 16-byte vectors per column: D / 8
  int32_t B, H, k, W_in;
  const int32_t* pad_in;
  const int32_t* n_acc;
  const int32_t* w_new;
  uint32_t* dev_status;
  uint32_t chunks;                       // workgroups per span (out of place)
  uint32_t misaligned;                   // out of place: spans tiled from the group boundary below them
  uint32_t realign_blocks;               // realign workgroups in this launch
  uint32_t span_base;                    // first span of this launch
  uint32_t nspans;                       // L * 2 * B * H
  // workgroups before the realign ones: position ids / mask, then the token row
  uint32_t extra_blocks;
  uint32_t pm_blocks;
  int64_t* pos;
  uint8_t* mask;
  const int32_t* pad_out;
  int64_t pm_cap;
  uint32_t pm_col_blocks;
  const int32_t* s_in;                   // token row S [B][s_in_stride]
  int32_t* s_out;                        // [B][s_out_stride]; == s_in: in place
  int64_t s_in_stride, s_out_stride;
  const int32_t* tokens;                 // [B][k+1] predictions from verification
  int32_t pad_id;
  uint32_t tok_col_blocks;               // workgroups per token row (1 in place)
  uint32_t tok_blocks;                   // token-row workgroups in all
  uint32_t* clear_words;                 // one more workgroup zeroes these (NULL: none)
  uint32_t clear_count;
  const int32_t* order;                  // in place: verification's order table (NULL: the cache's order)
  uint32_t span_rows;                    // spans per row: L * 2 * H
};

struct RowGeom {
  int32_t pad_in, pad_out, len, w;
};

__device__ __forceinline__ uint32_t row_geometry(const RealignArgs& a, int row, RowGeom& g) {
  const int32_t L = a.W_in - (a.k + 1);
  const int32_t w = load_invariant(a.w_new);
  const int32_t p = load_invariant(a.pad_in + row);
  const int32_t n = load_invariant(a.n_acc + row);
  uint32_t err = 0u;
  if (p < 0 || p > L) err |= kBadPadIn;
  if (n < 0 || n > a.k) err |= kBadAccept;
  if (err) return err;
  const int32_t len = (L - p) + n + 1;
  if (w < 1 || w > a.W_in || len > w) return kBadWidth;
  g.pad_in = p;
  g.pad_out = w - len;
  g.len = len;
  g.w = w;
  return 0u;
}

// Position ids and mask for 4*kTpb columns of one row.
template <int kTpb>
__device__ void posmask_block(uint32_t blk, int64_t* pos, uint8_t* mask, const int32_t* pad_out,
                              const int32_t* w_new, int32_t k, int64_t pm_cap, uint32_t col_blocks,
                              uint32_t* dev_status) {
  const uint32_t row = blk / col_blocks;
  const uint32_t cb = blk - row * col_blocks;
  const int32_t w = load_invariant(w_new);
  const int32_t po = load_invariant(pad_out + row);
  const int64_t width = static_cast<int64_t>(w) + k + 1;
  if (w < 0 || po < 0 || po > w || width > pm_cap) {
    if (cb == 0 && threadIdx.x == 0 && dev_status) atomicOr(dev_status, kBadPadOut);
    return;
  }
  posmask_cols<kTpb>(cb, pos + static_cast<int64_t>(row) * pm_cap, mask + static_cast<int64_t>(row) * pm_cap, po,
                     width);
}

// Token row S of one sequence (Alg. 1, phase 3): the c_i + 1 tokens of the
// row (its cached tokens and the pending token) move from column pad_in to
// pad_out, the accepted drafts and the bonus token (the predictions
// tokens[0..n_acc]) follow them, and columns [0, pad_out) hold pad_id; the
// new row is L' + 1 wide.  Out of place a workgroup writes 4*kTpb columns of
// one row; in place one workgroup walks the whole row in the direction of its
// shift and writes the padding and the appended tokens after a barrier.
template <int kTpb>
__device__ void token_block(const RealignArgs& a, uint32_t blk) {
  const uint32_t row = blk / a.tok_col_blocks;
  const uint32_t cb = blk - row * a.tok_col_blocks;
  const int32_t L = a.W_in - (a.k + 1);
  const int32_t w = load_invariant(a.w_new);
  const int32_t p = load_invariant(a.pad_in + row);
  const int32_t n = load_invariant(a.n_acc + row);
  uint32_t err = 0u;
  if (p < 0 || p > L) err |= kBadPadIn;
  if (n < 0 || n > a.k) err |= kBadAccept;
  const int32_t c = L - p;
  if (!err && (w < 1 || w > a.W_in || c + n + 1 > w)) err |= kBadWidth;
  if (err) {
    if (cb == 0 && threadIdx.x == 0 && a.dev_status) atomicOr(a.dev_status, err);
    return;
  }
  const int64_t po = static_cast<int64_t>(w) - (c + n + 1);   // new padding
  const int64_t keep_end = po + c + 1;                          // end of the moved tokens
  const int64_t width = static_cast<int64_t>(w) + 1;
  const int32_t* src = a.s_in + static_cast<int64_t>(row) * a.s_in_stride;
  int32_t* dst = a.s_out + static_cast<int64_t>(row) * a.s_out_stride;
  const int32_t* tk = a.tokens + static_cast<int64_t>(row) * (a.k + 1);
  if (a.s_in != a.s_out) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t j = static_cast<int64_t>(cb) * (4 * kTpb) + q * kTpb + threadIdx.x;
      if (j < width) {
        int32_t v;
        if (j < po) v = a.pad_id;
        else if (j < keep_end) v = src[j - po + p];
        else v = tk[j - keep_end];
        dst[j] = v;
      }
    }
    return;
  }
  // in place
  const int64_t nt = c + 1;
  const int64_t shift = po - p;
  constexpr int64_t kChunk = 4 * kTpb;
  if (shift != 0) {
    for (int64_t it = 0; it < nt; it += kChunk) {
      // right shifts walk from the top, left shifts from the bottom
      const int64_t lo = shift > 0 ? nt - it - kChunk : it;
      int32_t v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int64_t u = lo + q * kTpb + threadIdx.x;
        u = u < 0 ? 0 : (u >= nt ? nt - 1 : u);
        v[q] = dst[p + u];
      }
      asm volatile("" ::"v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3]));
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t u = lo + q * kTpb + threadIdx.x;
        if (u >= 0 && u < nt) dst[po + u] = v[q];
      }
    }
    __syncthreads();
  }
  for (int64_t j = threadIdx.x; j < po; j += kTpb) dst[j] = a.pad_id;
  for (int64_t j = keep_end + threadIdx.x; j < width; j += kTpb) dst[j] = tk[j - keep_end];
}

template <int kTpb>
__device__ __forceinline__ void extra_block(const RealignArgs& a, uint32_t b) {
  if (b < a.pm_blocks)
    posmask_block<kTpb>(b, a.pos, a.mask, a.pad_out, a.w_new, a.k, a.pm_cap, a.pm_col_blocks, a.dev_status);
  else if (b - a.pm_blocks < a.tok_blocks)
    token_block<kTpb>(a, b - a.pm_blocks);
  else   // the completion counts of the one-launch verification that ran before
    for (uint32_t q = threadIdx.x; q < a.clear_count; q += kTpb) a.clear_words[q] = 0u;
}

// Out of place: the output of a span is cut into groups of kPieces*kSplit
// vectors, each covered by kSplit/kTpb workgroups; every workgroup moves
// kPieces pieces of one wave-width (see split_pieces).
template <int kPieces, int kTpb, int kSplit, int kNt>
__global__ __launch_bounds__(kTpb) void realign_oop_kernel(RealignArgs a) {
  if (blockIdx.x < a.extra_blocks) {
    extra_block<kTpb>(a, blockIdx.x);
    return;
  }
  const uint32_t b = blockIdx.x - a.extra_blocks;
  const uint32_t rel = b / a.chunks;
  const uint32_t sub = b - rel * a.chunks;            // workgroup within the span
  const uint32_t span = a.span_base + rel;
  const int row = static_cast<int>((span / static_cast<uint32_t>(a.H)) % static_cast<uint32_t>(a.B));
  RowGeom g;
  const uint32_t err = row_geometry(a, row, g);
  if (err) {
    if (sub == 0 && span == static_cast<uint32_t>(row) * a.H && threadIdx.x == 0 && a.dev_status)
      atomicOr(a.dev_status, err);
    return;
  }
  u32x4* dspan = a.dst + static_cast<int64_t>(span) * a.dst_span_vecs;
  const int64_t mis = a.misaligned ? split_misalign<kPieces, kSplit>(dspan) : 0;
  const int64_t base = split_base<kPieces, kTpb, kSplit>(sub) - mis;
  const int64_t vpc = a.vpc;
  const int64_t total = static_cast<int64_t>(g.w) * vpc;        // output vectors of the span
  if (base >= total) return;
  const int64_t zero_end = static_cast<int64_t>(g.pad_out) * vpc;
  const int64_t shift = static_cast<int64_t>(g.pad_out - g.pad_in) * vpc;
  split_pieces<kPieces, kTpb, kSplit, kNt>(a.src + static_cast<int64_t>(span) * a.src_span_vecs, dspan, base, total,
                                           zero_end, shift);
}

// Register values of the current thread are live; forces the compiler to
// wait for the loads that produce them before this point.
__device__ __forceinline__ void hold(const u32x4& v) {
  asm volatile("" ::"v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w));
}

// Loads chunk [lo, lo + kTpb*kVec) (clipped to [0, n); indices outside are
// clamped, their values unused) of one row's kept vectors, which start at
// `from` within the span.
template <int kVec, int kTpb, int kNt>
__device__ __forceinline__ void load_chunk(const u32x4* base, int64_t from, int64_t lo, int64_t n, u32x4 (&v)[kVec]) {
  const int64_t t0 = static_cast<int64_t>(threadIdx.x >> 6) * (64 * kVec) + (threadIdx.x & 63);
#pragma unroll
  for (int j = 0; j < kVec; ++j) {
    int64_t u = lo + t0 + j * 64;
    u = u < 0 ? 0 : (u >= n ? n - 1 : u);
    v[j] = ld16<(kNt & 1) != 0>(base + (from + u));
  }
}

template <int kVec, int kTpb, int kNt>
__device__ __forceinline__ void store_chunk(u32x4* base, int64_t to, int64_t lo, int64_t n, const u32x4 (&v)[kVec]) {
  const int64_t w0 = lo + static_cast<int64_t>(wave_index()) * (64 * kVec);   // the wave's first vector
  const int lane = static_cast<int>(threadIdx.x & 63);
  u32x4* wb = base + (to + w0);
#pragma unroll
  for (int j = 0; j < kVec; ++j) {
    const int64_t u = w0 + lane + j * 64;
    if (u >= 0 && u < n) st16_at<(kNt & 2) != 0>(wb, static_cast<uint32_t>(lane + j * 64), v[j]);
  }
}

// Workgroup barrier that orders nothing but execution: the values this
// thread loaded are already in its registers (hold), so no other thread's
// later store can change them; loads issued after the barrier's program point
// stay in flight across it.
__device__ __forceinline__ void exec_barrier() { asm volatile("s_barrier" ::: "memory"); }

// In place: one workgroup per span moves the row's kept vectors [from, from+n)
// to [to, to+n) in chunks of kTpb*kVec, walking from the top for a shift to
// higher addresses and from the bottom for a shift to lower ones.  The next
// chunk's source never meets the current chunk's destination, so its loads
// are issued before the current chunk is stored; a barrier after the current
// chunk's loads have landed keeps every read of a chunk ahead of every write
// to it.
template <int kVec, int kTpb, int kNt>
__global__ __launch_bounds__(kTpb) void realign_inplace_kernel(RealignArgs a) {
  if (blockIdx.x < a.extra_blocks) {
    extra_block<kTpb>(a, blockIdx.x);
    return;
  }
  // Workgroups are dispatched round-robin over the 8 XCDs, and only the rows
  // whose padding changes do any work.  In the cache's own order a row's H
  // spans sit on H consecutive workgroups: with H = 4 and every other row
  // moving, all the work would land on half the XCDs.  So workgroups take
  // the spans in groups of 8 consecutive spans (memory locality as in the
  // cache's order), with the group's spans rotated over the XCDs by the
  // group index: any periodic pattern of moving rows spreads over all XCDs.
  const uint32_t rel = a.span_base + (blockIdx.x - a.extra_blocks);
  const uint32_t grp = rel >> 3;
  const uint32_t lin =
      static_cast<uint64_t>(grp) * 8u + 8u <= a.nspans ? (grp << 3) + ((rel + grp) & 7u) : rel;
  uint32_t span;
  RowGeom g;
  if (a.order) {
    // the rows in the order verification wrote (longest moving rows first),
    // kInRowGroup rows at a time, each group slab by slab in the cache's
    // order: the index alone gives (group, slab, row, head), and one load the
    // row's geometry
    const uint32_t B = static_cast<uint32_t>(a.B), H = static_cast<uint32_t>(a.H);
    // R <= B, so a group's spans (R * span_rows <= nspans) fit 32 bits
    const uint32_t R = kInRowGroup && kInRowGroup < B ? kInRowGroup : B;   // 0: the whole batch is one group
    const uint32_t grp_spans = R * a.span_rows;
    const uint32_t gi = lin / grp_spans;
    const uint32_t rem = lin - gi * grp_spans;
    const uint32_t rows_here = B - gi * R < R ? B - gi * R : R;
    const uint32_t slab = rem / (rows_here * H);
    const uint32_t rr = rem - slab * rows_here * H;
    const uint32_t r = rr / H, h = rr - r * H;
    const int32_t* info = a.order + 4 * static_cast<int64_t>(gi * R + r);
    const uint32_t row_u = static_cast<uint32_t>(load_invariant(info));
    g.pad_in = load_invariant(info + 1);
    g.pad_out = load_invariant(info + 2);
    g.len = load_invariant(info + 3);
    span = (slab * B + row_u) * H + h;
  } else {
    span = lin;
    const uint32_t row_u = (span / static_cast<uint32_t>(a.H)) % static_cast<uint32_t>(a.B);
    const int row = static_cast<int>(row_u);
    const uint32_t err = row_geometry(a, row, g);
    if (err) {
      if (span == row_u * static_cast<uint32_t>(a.H) && threadIdx.x == 0 && a.dev_status) atomicOr(a.dev_status, err);
      return;
    }
  }
  const int32_t s = g.pad_out - g.pad_in;
  if (s == 0) return;  // no shift: the row is already in place (uniform acceptance)
  const int64_t vpc = a.vpc;
  u32x4* base = a.dst + static_cast<int64_t>(span) * a.dst_span_vecs;
  const int64_t n = static_cast<int64_t>(g.len) * vpc;
  const int64_t from = static_cast<int64_t>(g.pad_in) * vpc;
  const int64_t to = static_cast<int64_t>(g.pad_out) * vpc;
  constexpr int64_t kChunk = static_cast<int64_t>(kTpb) * kVec;
  const int64_t nchunks = (n + kChunk - 1) / kChunk;
  // chunk c starts at lo(c): from the top for s > 0, from the bottom for s < 0
  auto lo_of = [&](int64_t c) { return s > 0 ? n - (c + 1) * kChunk : c * kChunk; };
  u32x4 cur[kVec], nxt[kVec];
  load_chunk<kVec, kTpb, kNt>(base, from, lo_of(0), n, cur);
  for (int64_t c = 0; c < nchunks; ++c) {
    const bool more = c + 1 < nchunks;
    if (more) load_chunk<kVec, kTpb, kNt>(base, from, lo_of(c + 1), n, nxt);
#pragma unroll
    for (int j = 0; j < kVec; ++j) hold(cur[j]);
    exec_barrier();  // every thread's loads of chunk c have landed
    store_chunk<kVec, kTpb, kNt>(base, to, lo_of(c), n, cur);
    if (more) {
#pragma unroll
      for (int j = 0; j < kVec; ++j) cur[j] = nxt[j];
    }
  }
  if (s > 0) {
    // the vacated columns [pad_in, pad_out) become padding; every read of
    // them landed before the last barrier
    const u32x4 zero = {0u, 0u, 0u, 0u};
    for (int64_t u0 = 0; u0 < to - from; u0 += kTpb) {
      const int64_t w0 = u0 + static_cast<int64_t>(wave_index()) * 64;
      const int lane = static_cast<int>(threadIdx.x & 63);
      if (w0 + lane < to - from) st16_at<(kNt & 2) != 0>(base + (from + w0), static_cast<uint32_t>(lane), zero);
    }
  }
  // columns [0, pad_out) already hold padding (+0.0) for a shift to lower addresses
}

__global__ __launch_bounds__(kThreads) void posmask_kernel(int64_t* pos, uint8_t* mask,
                                                           const int32_t* pad_out, const int32_t* w_new,
                                                           int32_t k, int64_t pm_cap, uint32_t col_blocks,
                                                           uint32_t* dev_status) {
  posmask_block<kThreads>(blockIdx.x, pos, mask, pad_out, w_new, k, pm_cap, col_blocks, dev_status);
}

__global__ __launch_bounds__(kThreads) void tokens_kernel(RealignArgs a) {
  token_block<kThreads>(a, blockIdx.x);
}

__global__ __launch_bounds__(kThreads) void zero_kernel(uint4* p16, int64_t n16, uint8_t* tail, int64_t ntail) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (i < n16) p16[i] = make_uint4(0u, 0u, 0u, 0u);
  if (i < ntail) tail[i] = 0;
}

constexpr int kOopVec = SPECDEC_OOP_VEC, kOopTpb = SPECDEC_OOP_TPB, kOopNt = SPECDEC_OOP_NT;
constexpr int kOopSplit = SPECDEC_OOP_SPLIT;
constexpr int kInVec = SPECDEC_INPLACE_VEC, kInTpb = SPECDEC_INPLACE_TPB, kInNt = SPECDEC_INPLACE_NT;
static_assert(kOopTpb % 64 == 0 && kInTpb % 64 == 0, "workgroups are whole wavefronts");

}  // namespace

int64_t max_launch_items() {
  int64_t max_items = 0xFFFFFFFFLL;
  if (const char* env = std::getenv("SPECDEC_MAX_LAUNCH_ITEMS")) {
    const long long v = std::atoll(env);
    if (v > 0 && v < max_items) max_items = v;
  }
  return max_items;
}

int64_t verify_chunk_elems(int64_t rows, int64_t V) {
  // about SPECDEC_VERIFY_TARGET workgroups in total, each scanning
  // SPECDEC_VERIFY_MIN_CHUNK..SPECDEC_VERIFY_MAX_CHUNK elements (a multiple
  // of the minimum), and at most kMaxVerifyChunks workgroups per row
  constexpr int64_t kTarget = SPECDEC_VERIFY_TARGET, kMin = SPECDEC_VERIFY_MIN_CHUNK, kMax = SPECDEC_VERIFY_MAX_CHUNK;
  static_assert(kMin % 8 == 0 && kMax % kMin == 0, "chunks are whole 16-byte vectors");
  const int64_t per = (rows * V + kTarget - 1) / kTarget;
  int64_t c = ((per + kMin - 1) / kMin) * kMin;
  if (c < kMin) c = kMin;
  if (c > kMax) c = kMax;
  int64_t min_c = (V + kMaxVerifyChunks - 1) / kMaxVerifyChunks;
  min_c = ((min_c + 7) / 8) * 8;
  if (c < min_c) c = min_c;
  if (c > V) c = V;
  return c;
}

int64_t verify_chunks(int64_t rows, int64_t V) {
  const int64_t c = verify_chunk_elems(rows, V);
  return (V + c - 1) / c;
}

static VerifyArgs verify_args(const VerifyLaunch& p) {
  VerifyArgs a;
  a.logits = static_cast<const char*>(p.logits);
  a.draft = p.draft;
  a.pad_in = p.pad_in;
  a.B = p.B;
  a.k = p.k;
  a.V = p.V;
  a.W_in = p.W_in;
  a.tokens = p.tokens;
  a.n_acc = p.n_acc;
  a.bonus = p.bonus;
  a.pad_out = p.pad_out;
  a.w_new = p.w_new;
  a.partial = reinterpret_cast<unsigned long long*>(static_cast<char*>(p.workspace) + kWsHeaderBytes);
  a.dev_status = p.dev_status;
  const int64_t rows = static_cast<int64_t>(p.B) * (p.k + 1);
  a.chunk_elems = verify_chunk_elems(rows, p.V);
  a.chunks = static_cast<int32_t>((p.V + a.chunk_elems - 1) / a.chunk_elems);
  a.order = p.write_order ? reinterpret_cast<int32_t*>(static_cast<char*>(p.workspace) + order_offset(p.B, p.k, p.V))
                          : nullptr;
  return a;
}

int64_t order_offset(int64_t B, int64_t k, int64_t V) {
  const int64_t rows = B * (k + 1);
  return static_cast<int64_t>(kWsHeaderBytes) + ((rows * verify_chunks(rows, V) * 8 + 15) / 16) * 16;
}

int64_t order_bytes(int64_t B) { return 16 * B; }

hipError_t launch_verify_scan(const VerifyLaunch& p, hipStream_t stream) {
  const VerifyArgs a = verify_args(p);
  const int64_t blocks = static_cast<int64_t>(p.B) * (p.k + 1) * a.chunks;
  const dim3 grid(static_cast<uint32_t>(blocks)), block(kThreads);
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(verify_partial_kernel<0>, grid, block, 0, stream, a); break;
    case 1: hipLaunchKernelGGL(verify_partial_kernel<1>, grid, block, 0, stream, a); break;
    default: hipLaunchKernelGGL(verify_partial_kernel<2>, grid, block, 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_verify_finalize(const VerifyLaunch& p, hipStream_t stream) {
  const VerifyArgs a = verify_args(p);
  hipLaunchKernelGGL(verify_finalize_kernel, dim3(1), dim3(kFinalizeThreads), 0, stream, a);
  return hipGetLastError();
}

bool verify_fused_fits(int64_t B, int64_t k, int64_t V, int dtype) {
  const int64_t eb = dtype == 0 ? 4 : 2;
  return B >= 1 && B * (k + 1) <= kMaxFusedVerifyRows && V * eb <= kMaxFusedVerifyRowBytes;
}

hipError_t launch_verify_fused(const VerifyLaunch& p, uint32_t* counts, hipStream_t stream) {
  FusedVerifyArgs f;
  f.v = verify_args(p);
  // the counts first (cleared after the call), the lengths above every count
  // a batch of any size uses, so that no call's lengths land in another's counts
  f.batch_count = counts;
  f.seq_count = counts + 1;
  f.lens = reinterpret_cast<int32_t*>(counts + 1 + kMaxFusedVerifyRows);
  const dim3 grid(static_cast<uint32_t>(static_cast<int64_t>(p.B) * (p.k + 1))), block(kFusedThreads);
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(verify_fused_kernel<0>, grid, block, 0, stream, f); break;
    case 1: hipLaunchKernelGGL(verify_fused_kernel<1>, grid, block, 0, stream, f); break;
    default: hipLaunchKernelGGL(verify_fused_kernel<2>, grid, block, 0, stream, f); break;
  }
  return hipGetLastError();
}

hipError_t launch_verify(const VerifyLaunch& p, hipStream_t stream) {
  const hipError_t e = launch_verify_scan(p, stream);
  if (e != hipSuccess) return e;
  return launch_verify_finalize(p, stream);
}

static void fill_token_args(RealignArgs& a, const RealignLaunch& p, int tpb) {
  a.s_in = p.s_in;
  a.s_out = p.s_out;
  a.s_in_stride = p.s_in_stride;
  a.s_out_stride = p.s_out_stride;
  a.tokens = p.tokens;
  a.pad_id = p.pad_id;
  a.tok_col_blocks = 0;
  a.clear_words = p.clear_words;
  a.clear_count = p.clear_words ? p.clear_count : 0u;
  if (p.s_in) {
    const int64_t width = static_cast<int64_t>(p.W_in) + 1;   // L' + 1 <= W_in + 1
    a.tok_col_blocks = p.s_in == p.s_out ? 1u : static_cast<uint32_t>((width + 4 * tpb - 1) / (4 * tpb));
  }
}

hipError_t launch_realign(const RealignLaunch& p, hipStream_t stream) {
  RealignArgs a{};
  a.src = static_cast<const u32x4*>(p.src);
  a.dst = static_cast<u32x4*>(p.dst);
  a.vpc = p.D / 8;
  a.src_span_vecs = p.src_cap * a.vpc;
  a.dst_span_vecs = p.dst_cap * a.vpc;
  a.B = p.B;
  a.H = p.H;
  a.k = p.k;
  a.W_in = p.W_in;
  a.pad_in = p.pad_in;
  a.n_acc = p.n_acc;
  a.w_new = p.w_new;
  a.dev_status = p.dev_status;
  const int64_t nspans = static_cast<int64_t>(p.L) * 2 * p.B * p.H;
  a.nspans = static_cast<uint32_t>(nspans);
  a.pos = p.pos;
  a.mask = p.mask;
  a.pad_out = p.pad_out;
  a.pm_cap = p.pm_cap;
  a.order = p.in_place ? p.order : nullptr;
  a.span_rows = static_cast<uint32_t>(static_cast<int64_t>(p.L) * 2 * p.H);
  const int tpb = p.in_place ? kInTpb : kOopTpb;
  int64_t pm_blocks = 0;
  a.pm_col_blocks = 1;
  if (p.pos) {
    const int64_t bound = static_cast<int64_t>(p.W_in) + p.k + 1;
    a.pm_col_blocks = static_cast<uint32_t>((bound + 4 * tpb - 1) / (4 * tpb));
    pm_blocks = static_cast<int64_t>(a.pm_col_blocks) * p.B;
  }
  fill_token_args(a, p, tpb);
  const int64_t tok_blocks = static_cast<int64_t>(a.tok_col_blocks) * p.B;
  a.tok_blocks = static_cast<uint32_t>(tok_blocks);
  const int64_t extra = pm_blocks + tok_blocks + (a.clear_words ? 1 : 0);
  a.misaligned = !p.in_place && !split_spans_aligned<kOopVec, kOopSplit>(p.dst, a.dst_span_vecs);
  const int64_t chunks = p.in_place ? 1 : split_blocks<kOopVec, kOopTpb, kOopSplit>(
                                                static_cast<int64_t>(p.W_in) * a.vpc, a.misaligned != 0);
  a.chunks = static_cast<uint32_t>(chunks);
  // one dispatch holds fewer than 2^32 work-items: split the spans over
  // several launches when the cache is larger than that
  const int64_t max_blocks = (max_launch_items() / tpb) - extra;
  const int64_t spans_per_launch = max_blocks / chunks;
  if (spans_per_launch < 1) return hipErrorInvalidConfiguration;
  const dim3 block(tpb);
  for (int64_t s0 = 0; s0 < nspans || (nspans == 0 && s0 == 0); s0 += spans_per_launch) {
    const int64_t ns = nspans - s0 < spans_per_launch ? nspans - s0 : spans_per_launch;
    const bool first = s0 == 0;
    a.span_base = static_cast<uint32_t>(s0);
    a.realign_blocks = static_cast<uint32_t>(ns * chunks);
    a.extra_blocks = first ? static_cast<uint32_t>(extra) : 0u;
    a.pm_blocks = first ? static_cast<uint32_t>(pm_blocks) : 0u;
    const int64_t blocks = ns * chunks + (first ? extra : 0);
    if (blocks == 0) break;
    const dim3 grid(static_cast<uint32_t>(blocks));
    if (p.in_place)
      hipLaunchKernelGGL((realign_inplace_kernel<kInVec, kInTpb, kInNt>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((realign_oop_kernel<kOopVec, kOopTpb, kOopSplit, kOopNt>), grid, block, 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (nspans == 0) break;
  }
  return hipSuccess;
}

hipError_t launch_tokens(const RealignLaunch& p, hipStream_t stream) {
  RealignArgs a{};
  a.B = p.B;
  a.k = p.k;
  a.W_in = p.W_in;
  a.pad_in = p.pad_in;
  a.n_acc = p.n_acc;
  a.w_new = p.w_new;
  a.dev_status = p.dev_status;
  fill_token_args(a, p, kThreads);
  const int64_t blocks = static_cast<int64_t>(a.tok_col_blocks) * p.B;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(tokens_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}


hipError_t launch_posmask(const PosmaskLaunch& p, hipStream_t stream) {
  const int64_t col_blocks = (p.col_bound + kPmColsPerBlock - 1) / kPmColsPerBlock;
  const int64_t blocks = col_blocks * p.B;
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(posmask_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), 0, stream, p.pos,
                     p.mask, p.pad_out, p.w_new, p.k, p.pm_cap, static_cast<uint32_t>(col_blocks), p.dev_status);
  return hipGetLastError();
}

hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream) {
  const uintptr_t base = reinterpret_cast<uintptr_t>(ptr);
  // 16-byte stores over the aligned body, byte stores for the rest (the
  // workspace is 8-byte aligned; the rare unaligned prefix is byte-cleared)
  if ((base & 15u) != 0u || bytes < 16) {
    const int64_t n = static_cast<int64_t>(bytes);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(zero_kernel, dim3(static_cast<uint32_t>((n + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       stream, static_cast<uint4*>(nullptr), int64_t{0}, static_cast<uint8_t*>(ptr), n);
    return hipGetLastError();
  }
  const int64_t n16 = static_cast<int64_t>(bytes / 16);
  const int64_t ntail = static_cast<int64_t>(bytes % 16);
  const int64_t n = n16 > ntail ? n16 : ntail;
  hipLaunchKernelGGL(zero_kernel, dim3(static_cast<uint32_t>((n + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     stream, static_cast<uint4*>(ptr), n16, static_cast<uint8_t*>(ptr) + n16 * 16, ntail);
  return hipGetLastError();
}

}  // namespace specdec
