// HIP kernels of stochastic (temperature T > 0) verification on MI355X
// (gfx950, wave64): speculative sampling over a batch, the T > 0 counterpart of
// greedy BatchVerify (arXiv 2510.22876, Algorithm 3; the target-distribution
// requirement of output equivalence at T > 0).
//
//   sample_stats    every target and draft logit row, split over workgroups:
//                   the row maximum and the sum of exp((x - max) / T) of each
//                   chunk (online: a thread rescales its sum when its maximum
//                   grows), stored per chunk.
//   sample_mass     one workgroup per (sequence, chunk): merges the chunk
//                   statistics into the normalisers of p_r = softmax(target_r
//                   / T) and q_r = softmax(draft_r / T), accepts draft r iff
//                   u_r * q_r(x_r) < p_r(x_r) (wave 0, one lane per draft,
//                   first rejection by ballot; every chunk of a sequence
//                   takes the same decision), then sums the chunk's weights of
//                   the distribution to sample: the residual max(0, p_j - q_j)
//                   after a rejection at j (and p_j, its fallback), p_k after
//                   k acceptances.
//   sample_pick     one workgroup per sequence: inversion with u_sample over
//                   the chunk totals (a prefix over at most 64 chunks in wave
//                   0), then a tiled prefix scan of the one chunk where the
//                   running mass crosses u * total.
//   sample_width    one workgroup: new width and paddings (Eq. (1), Eq. (2)).
//
// Arithmetic is fp32 with exp2 of (x - max) * log2(e) / T; everything is
// bandwidth- or latency-bound, no matrix cores.
#include "specdec_internal.h"

namespace specdec {
namespace {

constexpr uint32_t kBadPadIn = 0x1u, kBadUniform = 0x40u;
constexpr int kStatsThreads = 256;
constexpr int kGroup = 8;                      // logits per thread per load (16 bytes of bf16 / f16)
constexpr float kLowest = -3.402823466e38f;    // start of a running maximum (finite, so -inf logits give 0)

template <int DT>
__device__ __forceinline__ float widen(const char* row, int64_t v) {
  if constexpr (DT == 0) {
    return *reinterpret_cast<const float*>(row + 4 * v);
  } else if constexpr (DT == 1) {
    const uint32_t u = static_cast<uint32_t>(*reinterpret_cast<const uint16_t*>(row + 2 * v)) << 16;
    return __uint_as_float(u);
  } else {
    return static_cast<float>(*reinterpret_cast<const _Float16*>(row + 2 * v));
  }
}

// Logits [8g, 8g + 8) of a row (clipped to V; missing ones are -inf), with one
// 16-byte load per four fp32 or eight 16-bit logits when the group is aligned.
template <int DT>
__device__ __forceinline__ void load_group(const char* row, int64_t g, int64_t V, bool aligned, float (&x)[kGroup]) {
  const int64_t e0 = g * kGroup;
  if (aligned && e0 + kGroup <= V) {
    if constexpr (DT == 0) {
      const uint4* p = reinterpret_cast<const uint4*>(row + 4 * e0);
      const uint4 a = p[0], b = p[1];
      x[0] = __uint_as_float(a.x); x[1] = __uint_as_float(a.y); x[2] = __uint_as_float(a.z); x[3] = __uint_as_float(a.w);
      x[4] = __uint_as_float(b.x); x[5] = __uint_as_float(b.y); x[6] = __uint_as_float(b.z); x[7] = __uint_as_float(b.w);
    } else {
      const uint4 a = *reinterpret_cast<const uint4*>(row + 2 * e0);
      const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if constexpr (DT == 1) {
          x[2 * q] = __uint_as_float(w[q] << 16);
          x[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
        } else {
          x[2 * q] = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w[q] & 0xFFFFu)));
          x[2 * q + 1] = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w[q] >> 16)));
        }
      }
    }
    return;
  }
#pragma unroll
  for (int e = 0; e < kGroup; ++e) x[e] = e0 + e < V ? widen<DT>(row, e0 + e) : -__builtin_inff();
}

__device__ __forceinline__ bool row_aligned(const char* row, int eb) {
  return (reinterpret_cast<uintptr_t>(row) & 15u) == 0 && eb * kGroup % 16 == 0;
}

struct SampleArgs {
  const char* logits;        // [B][k+1][V]
  const char* draft_logits;  // [B][k][V]
  const int32_t* draft;
  const int32_t* pad_in;
  const float* u_accept;     // [B][k]
  const float* u_sample;     // [B]
  float c;                   // log2(e) / T
  int32_t B, k, V, W_in;
  int32_t* tokens;
  int32_t* n_acc;
  int32_t* bonus;
  int32_t* pad_out;
  int32_t* w_new;
  float2* partial;           // [B*(2k+1)][chunks]: (max, sum of exp2((x - max) * c))
  float2* mass;              // [B][chunks]: (residual weight, target weight) of each chunk
  int2* last;                // [B][chunks]: last index of positive residual / target weight
  uint32_t* dev_status;
  int64_t chunk_elems;       // a multiple of kGroup, or V (one chunk)
  int32_t chunks;
};

// Row rho < B*(k+1) is target row rho; the rest are draft rows.
template <int DT>
__device__ __forceinline__ const char* stats_row(const SampleArgs& a, int64_t rho) {
  constexpr int eb = DT == 0 ? 4 : 2;
  const int64_t nt = static_cast<int64_t>(a.B) * (a.k + 1);
  return rho < nt ? a.logits + rho * a.V * eb : a.draft_logits + (rho - nt) * a.V * eb;
}

__device__ __forceinline__ void merge(float& m, float& s, float m2, float s2, float c) {
  const float mm = fmaxf(m, m2);
  s = s * exp2f((m - mm) * c) + s2 * exp2f((m2 - mm) * c);
  m = mm;
}

template <int DT>
__global__ __launch_bounds__(kStatsThreads) void sample_stats_kernel(SampleArgs a) {
  constexpr int eb = DT == 0 ? 4 : 2;
  __shared__ float wm[kStatsThreads / 64], ws[kStatsThreads / 64];
  const int64_t rho = blockIdx.x / a.chunks;
  const int64_t chunk = blockIdx.x - rho * a.chunks;
  const char* row = stats_row<DT>(a, rho);
  const bool aligned = row_aligned(row, eb);
  const int64_t beg = chunk * a.chunk_elems;
  int64_t end = beg + a.chunk_elems;
  if (end > a.V) end = a.V;
  float m = kLowest, s = 0.0f;
  for (int64_t g = beg / kGroup + threadIdx.x; g * kGroup < end; g += kStatsThreads) {
    float x[kGroup];
    load_group<DT>(row, g, end, aligned, x);
    float gm = x[0];
#pragma unroll
    for (int e = 1; e < kGroup; ++e) gm = fmaxf(gm, x[e]);
    if (gm > m) {
      s *= exp2f((m - gm) * a.c);
      m = gm;
    }
#pragma unroll
    for (int e = 0; e < kGroup; ++e) s += exp2f((x[e] - m) * a.c);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) merge(m, s, __shfl_xor(m, off), __shfl_xor(s, off), a.c);
  if ((threadIdx.x & 63) == 0) {
    wm[threadIdx.x >> 6] = m;
    ws[threadIdx.x >> 6] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = wm[0], S = ws[0];
#pragma unroll
    for (int q = 1; q < kStatsThreads / 64; ++q) merge(M, S, wm[q], ws[q], a.c);
    a.partial[blockIdx.x] = make_float2(M, S);
  }
}

// Normalisers of sequence i's rows into LDS: slot r <= k is target row r,
// slot k+1+r draft row r (the chunk statistics merged in chunk order).
__device__ __forceinline__ void row_norms(const SampleArgs& a, int i, float* rowM, float* rowS) {
  const int k = a.k;
  const int64_t nt = static_cast<int64_t>(a.B) * (k + 1);
  for (int t = threadIdx.x; t < 2 * k + 1; t += blockDim.x) {
    const int64_t rho = t <= k ? static_cast<int64_t>(i) * (k + 1) + t : nt + static_cast<int64_t>(i) * k + (t - k - 1);
    const float2* p = a.partial + rho * a.chunks;
    float M = p[0].x, S = p[0].y;
    for (int q = 1; q < a.chunks; ++q) merge(M, S, p[q].x, p[q].y, a.c);
    rowM[t] = M;
    rowS[t] = S;
  }
}

// Acceptance tests of sequence i, one lane of wave 0 per draft: draft r is
// accepted iff u_r * q_r(x_r) < p_r(x_r).  Returns (to wave 0) the first
// rejected slot, k if none.
template <int DT>
__device__ __forceinline__ int accepted_count(const SampleArgs& a, int i, const float* rowM, const float* rowS,
                                              bool flag) {
  constexpr int eb = DT == 0 ? 4 : 2;
  const int k = a.k;
  const int64_t V = a.V;
  bool reject = false;
  const int r = threadIdx.x;
  if (r < k) {
    float u = a.u_accept[static_cast<int64_t>(i) * k + r];
    if (!(u >= 0.0f && u < 1.0f)) {
      if (flag && a.dev_status) atomicOr(a.dev_status, kBadUniform);
      u = u >= 1.0f ? 0.99999994f : 0.0f;
    }
    const int32_t x = a.draft[static_cast<int64_t>(i) * k + r];
    float px = 0.0f, qx = 0.0f;
    if (x >= 0 && x < V) {
      const float lt = widen<DT>(a.logits + (static_cast<int64_t>(i) * (k + 1) + r) * V * eb, x);
      const float ld = widen<DT>(a.draft_logits + (static_cast<int64_t>(i) * k + r) * V * eb, x);
      px = exp2f((lt - rowM[r]) * a.c) / rowS[r];
      qx = exp2f((ld - rowM[k + 1 + r]) * a.c) / rowS[k + 1 + r];
    }
    reject = !(u * qx < px);
  }
  const unsigned long long rej = __ballot(reject);
  return rej ? __builtin_ctzll(rej) : k;
}

// The rows a sequence samples from after j accepted drafts: the residual
// max(0, p_j - q_j) when j < k (target row j, draft row j), else p_k; the
// target weight e = exp2((x - max) * c) is p_j unnormalised.
template <int DT>
struct SampleRows {
  const char* trow;
  const char* drow;
  float tM, tinv, dM, dinv;
  bool ta, da, residual;
  __device__ void init(const SampleArgs& a, int i, int j, const float* rowM, const float* rowS) {
    constexpr int eb = DT == 0 ? 4 : 2;
    const int k = a.k;
    residual = j < k;
    trow = a.logits + (static_cast<int64_t>(i) * (k + 1) + j) * a.V * eb;
    drow = residual ? a.draft_logits + (static_cast<int64_t>(i) * k + j) * a.V * eb : trow;
    tM = rowM[j];
    tinv = 1.0f / rowS[j];
    dM = residual ? rowM[k + 1 + j] : 0.0f;
    dinv = residual ? 1.0f / rowS[k + 1 + j] : 0.0f;
    ta = row_aligned(trow, eb);
    da = row_aligned(drow, eb);
  }
  // residual weights (0 when there is no residual) and target weights of a group
  __device__ __forceinline__ void weights(int64_t g, int64_t end, float c, float (&wr)[kGroup],
                                          float (&wp)[kGroup]) const {
    float xt[kGroup];
    load_group<DT>(trow, g, end, ta, xt);
#pragma unroll
    for (int e = 0; e < kGroup; ++e) wp[e] = exp2f((xt[e] - tM) * c);
    if (residual) {
      float xd[kGroup];
      load_group<DT>(drow, g, end, da, xd);
#pragma unroll
      for (int e = 0; e < kGroup; ++e) wr[e] = fmaxf(wp[e] * tinv - exp2f((xd[e] - dM) * c) * dinv, 0.0f);
    } else {
#pragma unroll
      for (int e = 0; e < kGroup; ++e) wr[e] = 0.0f;
    }
  }
};

constexpr int kMassThreads = 256;
constexpr int kPickThreads = 256;

// One workgroup per (sequence, chunk): the sequence's accepted count
// (recomputed by every chunk, identically), then the chunk's total residual
// and target weight and the last index of positive weight of each.
template <int DT>
__global__ __launch_bounds__(kMassThreads) void sample_mass_kernel(SampleArgs a) {
  __shared__ float rowM[2 * (64 + 1)], rowS[2 * (64 + 1)];
  __shared__ float redf[2][kMassThreads / 64];
  __shared__ int32_t redi[2][kMassThreads / 64];
  __shared__ int32_t s_nacc;
  const int i = static_cast<int>(blockIdx.x / a.chunks);
  const int64_t chunk = blockIdx.x - static_cast<int64_t>(i) * a.chunks;
  row_norms(a, i, rowM, rowS);
  __syncthreads();
  if (threadIdx.x < 64) {
    const int j = accepted_count<DT>(a, i, rowM, rowS, chunk == 0);
    if (threadIdx.x == 0) {
      s_nacc = j;
      if (chunk == 0) a.n_acc[i] = j;
    }
  }
  __syncthreads();
  SampleRows<DT> rows;
  rows.init(a, i, s_nacc, rowM, rowS);
  const int64_t beg = chunk * a.chunk_elems;
  int64_t end = beg + a.chunk_elems;
  if (end > a.V) end = a.V;
  float sr = 0.0f, sp = 0.0f;
  int32_t lr = -1, lp = -1;
  for (int64_t g = beg / kGroup + threadIdx.x; g * kGroup < end; g += kMassThreads) {
    float wr[kGroup], wp[kGroup];
    rows.weights(g, end, a.c, wr, wp);
#pragma unroll
    for (int e = 0; e < kGroup; ++e) {
      sr += wr[e];
      sp += wp[e];
      if (wr[e] > 0.0f) lr = static_cast<int32_t>(g * kGroup + e);
      if (wp[e] > 0.0f) lp = static_cast<int32_t>(g * kGroup + e);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    sr += __shfl_xor(sr, off);
    sp += __shfl_xor(sp, off);
    const int32_t o1 = __shfl_xor(lr, off), o2 = __shfl_xor(lp, off);
    lr = o1 > lr ? o1 : lr;
    lp = o2 > lp ? o2 : lp;
  }
  if ((threadIdx.x & 63) == 0) {
    redf[0][threadIdx.x >> 6] = sr;
    redf[1][threadIdx.x >> 6] = sp;
    redi[0][threadIdx.x >> 6] = lr;
    redi[1][threadIdx.x >> 6] = lp;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float tr = 0.0f, tp = 0.0f;
    int32_t mr = -1, mp = -1;
#pragma unroll
    for (int q = 0; q < kMassThreads / 64; ++q) {
      tr += redf[0][q];
      tp += redf[1][q];
      mr = redi[0][q] > mr ? redi[0][q] : mr;
      mp = redi[1][q] > mp ? redi[1][q] : mp;
    }
    a.mass[blockIdx.x] = make_float2(tr, tp);
    a.last[blockIdx.x] = make_int2(mr, mp);
  }
}

// Inclusive prefix sum over the block in thread order; *total gets the sum.
template <int kThreadsT>
__device__ __forceinline__ float block_inclusive_scan(float v, float* red, float* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  __syncthreads();
  if (lane == 63) red[wave] = v;
  __syncthreads();
  float before = 0.0f, all = 0.0f;
#pragma unroll
  for (int q = 0; q < kThreadsT / 64; ++q) {
    const float r = red[q];
    before += q < wave ? r : 0.0f;
    all += r;
  }
  *total = all;
  return before + v;
}

// One workgroup per sequence: inversion with u_sample over the chunk totals
// (wave 0: prefix over the chunks, the first chunk whose running total
// exceeds u * total), then a tiled scan of that chunk alone.  A residual with
// no mass falls back to p_j; where rounding leaves no crossing, the last
// index of positive weight is taken.
template <int DT>
__global__ __launch_bounds__(kPickThreads) void sample_pick_kernel(SampleArgs a) {
  __shared__ float rowM[2 * (64 + 1)], rowS[2 * (64 + 1)];
  __shared__ float red[kPickThreads / 64];
  __shared__ int32_t redl[kPickThreads / 64];
  __shared__ int32_t s_chunk, s_first, s_pick, s_fallback, s_use_res;
  __shared__ float s_excl, s_target;
  const int i = blockIdx.x;
  const int k = a.k;
  const int j = a.n_acc[i];
  row_norms(a, i, rowM, rowS);
  if (threadIdx.x < 64) {
    // chunk totals in chunk order, one lane per chunk (at most 64 chunks)
    const int c = threadIdx.x;
    const float2 m = c < a.chunks ? a.mass[static_cast<int64_t>(i) * a.chunks + c] : make_float2(0.0f, 0.0f);
    const int2 l = c < a.chunks ? a.last[static_cast<int64_t>(i) * a.chunks + c] : make_int2(-1, -1);
    float rtot = m.x;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) rtot += __shfl_xor(rtot, off);
    const bool use_res = j < k && rtot > 0.0f;
    float v = use_res ? m.x : m.y;
    int32_t lastpos = use_res ? l.x : l.y;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_up(v, off);
      if (c >= off) v += o;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(lastpos, off);
      lastpos = o > lastpos ? o : lastpos;
    }
    const float total = __shfl(v, 63);
    float us = a.u_sample[i];
    if (!(us >= 0.0f && us < 1.0f)) {
      if (c == 0 && a.dev_status) atomicOr(a.dev_status, kBadUniform);
      us = us >= 1.0f ? 0.99999994f : 0.0f;
    }
    const float target = us * total;
    const float prev = __shfl_up(v, 1);
    const unsigned long long hit = __ballot(c < a.chunks && v > target);
    if (c == 0) {
      const int cs = hit ? __builtin_ctzll(hit) : -1;
      s_chunk = cs;
      s_fallback = lastpos;
      s_use_res = use_res ? 1 : 0;
      s_target = target;
      s_pick = -1;
    }
    if (hit && c == __builtin_ctzll(hit)) s_excl = c == 0 ? 0.0f : prev;
  }
  __syncthreads();
  const int cs = s_chunk;
  if (cs >= 0) {
    SampleRows<DT> rows;
    rows.init(a, i, j, rowM, rowS);
    const bool use_res = s_use_res != 0;
    const float target = s_target;
    const int64_t beg = static_cast<int64_t>(cs) * a.chunk_elems;
    int64_t end = beg + a.chunk_elems;
    if (end > a.V) end = a.V;
    float running = s_excl;
    int32_t chunk_last = -1;
    for (int64_t g0 = beg / kGroup; g0 * kGroup < end; g0 += kPickThreads) {
      const int64_t g = g0 + threadIdx.x;
      float w[kGroup] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (g * kGroup < end) {
        float wr[kGroup], wp[kGroup];
        rows.weights(g, end, a.c, wr, wp);
#pragma unroll
        for (int e = 0; e < kGroup; ++e) w[e] = use_res ? wr[e] : wp[e];
      }
      float gs = 0.0f;
#pragma unroll
      for (int e = 0; e < kGroup; ++e) {
        gs += w[e];
        if (w[e] > 0.0f) chunk_last = static_cast<int32_t>(g * kGroup + e);
      }
      float tile = 0.0f;
      const float incl = running + block_inclusive_scan<kPickThreads>(gs, red, &tile);
      if (threadIdx.x == 0) s_first = 0x7FFFFFFF;
      __syncthreads();
      if (incl > target) atomicMin(&s_first, static_cast<int32_t>(threadIdx.x));
      __syncthreads();
      const int32_t first = s_first;
      if (first != 0x7FFFFFFF) {
        if (static_cast<int32_t>(threadIdx.x) == first) {
          float c = incl - gs;
          int32_t pick = -1, lastg = -1;
#pragma unroll
          for (int e = 0; e < kGroup; ++e) {
            c += w[e];
            if (pick < 0 && c > target && w[e] > 0.0f) pick = static_cast<int32_t>(g * kGroup + e);
            if (w[e] > 0.0f) lastg = static_cast<int32_t>(g * kGroup + e);
          }
          s_pick = pick >= 0 ? pick : lastg;
        }
        break;
      }
      running += tile;
    }
    // no crossing inside the chunk (rounding): the last positive weight the
    // scan saw in the chunk
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(chunk_last, off);
      chunk_last = o > chunk_last ? o : chunk_last;
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) redl[threadIdx.x >> 6] = chunk_last;
    __syncthreads();
    if (threadIdx.x == 0 && s_pick < 0) {
      int32_t m = -1;
#pragma unroll
      for (int q = 0; q < kPickThreads / 64; ++q) m = redl[q] > m ? redl[q] : m;
      s_pick = m;
    }
  }
  __syncthreads();
  int32_t x_out = s_pick;
  if (x_out < 0 || x_out >= a.V) x_out = s_fallback;
  if (threadIdx.x <= k) {
    const int r = threadIdx.x;
    a.tokens[static_cast<int64_t>(i) * (k + 1) + r] =
        r < j ? a.draft[static_cast<int64_t>(i) * k + r] : (r == j ? x_out : -1);
  }
  if (threadIdx.x == 0 && a.bonus) a.bonus[i] = x_out;
}

// New width and paddings (Eq. (1), Eq. (2)) from the accepted counts.
__global__ __launch_bounds__(1024) void sample_width_kernel(SampleArgs a) {
  __shared__ int32_t wmax[16];
  const int32_t L = a.W_in - (a.k + 1);
  int32_t local = 0;
  for (int i = threadIdx.x; i < a.B; i += 1024) {
    const int32_t p = a.pad_in[i];
    if (p >= 0 && p <= L) {
      const int32_t len = (L - p) + a.n_acc[i] + 1;
      local = len > local ? len : local;
    } else if (a.dev_status) {
      atomicOr(a.dev_status, kBadPadIn);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t o = __shfl_xor(local, off);
    local = o > local ? o : local;
  }
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = local;
  __syncthreads();
  int32_t w = wmax[0];
#pragma unroll
  for (int q = 1; q < 16; ++q) w = wmax[q] > w ? wmax[q] : w;
  for (int i = threadIdx.x; i < a.B; i += 1024) {
    const int32_t p = a.pad_in[i];
    a.pad_out[i] = (p >= 0 && p <= L) ? w - ((L - p) + a.n_acc[i] + 1) : -1;
  }
  if (threadIdx.x == 0) a.w_new[0] = w;
}

}  // namespace

int64_t sample_chunk_elems(int64_t rows, int64_t V) {
  int64_t c = verify_chunk_elems(rows, V);
  if (c < V) c = ((c + kGroup - 1) / kGroup) * kGroup;
  return c;
}

int64_t sample_chunks(int64_t rows, int64_t V) {
  const int64_t c = sample_chunk_elems(rows, V);
  return (V + c - 1) / c;
}

hipError_t launch_verify_sample(const SampleLaunch& p, hipStream_t stream) {
  SampleArgs a{};
  a.logits = static_cast<const char*>(p.logits);
  a.draft_logits = static_cast<const char*>(p.draft_logits);
  a.draft = p.draft;
  a.pad_in = p.pad_in;
  a.u_accept = p.u_accept;
  a.u_sample = p.u_sample;
  a.c = p.c;
  a.B = p.B;
  a.k = p.k;
  a.V = p.V;
  a.W_in = p.W_in;
  a.tokens = p.tokens;
  a.n_acc = p.n_acc;
  a.bonus = p.bonus;
  a.pad_out = p.pad_out;
  a.w_new = p.w_new;
  a.dev_status = p.dev_status;
  const int64_t rows = static_cast<int64_t>(p.B) * (2 * p.k + 1);
  a.chunk_elems = sample_chunk_elems(rows, p.V);
  a.chunks = static_cast<int32_t>((p.V + a.chunk_elems - 1) / a.chunk_elems);
  char* ws = static_cast<char*>(p.workspace) + kWsHeaderBytes;
  a.partial = reinterpret_cast<float2*>(ws);
  a.mass = reinterpret_cast<float2*>(ws + rows * a.chunks * 8);
  a.last = reinterpret_cast<int2*>(ws + (rows + p.B) * a.chunks * 8);
  const dim3 grid(static_cast<uint32_t>(rows * a.chunks));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_stats_kernel<0>, grid, dim3(kStatsThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_stats_kernel<1>, grid, dim3(kStatsThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_stats_kernel<2>, grid, dim3(kStatsThreads), 0, stream, a); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 mgrid(static_cast<uint32_t>(static_cast<int64_t>(p.B) * a.chunks));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_mass_kernel<0>, mgrid, dim3(kMassThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_mass_kernel<1>, mgrid, dim3(kMassThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_mass_kernel<2>, mgrid, dim3(kMassThreads), 0, stream, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 seqs(static_cast<uint32_t>(p.B));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_pick_kernel<0>, seqs, dim3(kPickThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_pick_kernel<1>, seqs, dim3(kPickThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_pick_kernel<2>, seqs, dim3(kPickThreads), 0, stream, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_width_kernel, dim3(1), dim3(1024), 0, stream, a);
  return hipGetLastError();
}

}  // namespace specdec
