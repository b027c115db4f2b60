// HIP kernels of stochastic (temperature T > 0) verification on MI355X
// (gfx950, wave64): speculative sampling over a batch, the T > 0 counterpart of
// greedy BatchVerify (arXiv 2510.22876, Algorithm 3; the target-distribution
// requirement of output equivalence at T > 0).
//
//   sample_stats    every target and draft logit row, split over workgroups:
//                   the row maximum and the sum of exp((x - max) / T) of each
//                   chunk (online: a thread rescales its sum when its maximum
//                   grows), stored per chunk.
//   sample_accept   one workgroup per sequence: merges the chunk statistics
//                   into the normalisers of p_r = softmax(target_r / T) and
//                   q_r = softmax(draft_r / T) (one wave per row), accepts
//                   draft r iff u_r * q_r(x_r) < p_r(x_r) (wave 0, one lane
//                   per draft, first rejection by ballot) and stores n_acc and
//                   the normalisers of the rows the sequence samples from.
//   sample_mass     one workgroup per (sequence, chunk of V/64 logits, at
//                   least 2048): the chunk's weights of the distribution to
//                   sample, the residual max(0, p_j - q_j) after a rejection
//                   at j (and p_j, its fallback), p_k after k acceptances.
//                   It also stores the weight total of every tile of 2048
//                   logits.
//   sample_pick     one workgroup per sequence: inversion with u_sample,
//                   coarse to fine: the chunk totals (a prefix over at most
//                   64 chunks in wave 0), the tile totals of the crossing
//                   chunk, then one block-wide scan of the crossing tile.
//                   Workgroup 0 also writes the new width and paddings
//                   (Eq. (1), Eq. (2)).
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
constexpr int kTile = 2048;                     // logits per sub-chunk total (one pick tile)

// 2^x with the hardware instruction (about 1 ulp; results below the normal
// range flush to 0, i.e. probabilities below 2^-126 of the row maximum's).
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

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
  float4* norms;             // [B]: (max, 1/sum) of the target and draft rows each sequence samples from
  float2* mass;              // [B][mchunks][tiles]: (residual weight, target weight) of each tile
  int2* last;                // [B][mchunks]: last index of positive residual / target weight
  int64_t mchunk_elems;      // logits per mass chunk (a multiple of kGroup, or V)
  int32_t mchunks;           // mass chunks per row (<= 64)
  int32_t tiles;             // tiles of kTile logits per mass chunk
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
  s = s * ex2((m - mm) * c) + s2 * ex2((m2 - mm) * c);
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
      s *= ex2((m - gm) * a.c);
      m = gm;
    }
#pragma unroll
    for (int e = 0; e < kGroup; ++e) s += ex2((x[e] - m) * a.c);
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

// Normaliser (max, sum) of one logit row from its chunk statistics, by one
// wave: lane q loads chunk q (all loads in flight at once; at most 64
// chunks), then a shuffle tree merges them.  Every kernel that needs a row's
// normaliser uses this, so they all get the same bits.
__device__ __forceinline__ float2 row_norm(const SampleArgs& a, int64_t rho) {
  const int lane = threadIdx.x & 63;
  float M = kLowest, S = 0.0f;
  if (lane < a.chunks) {
    const float2 p = a.partial[rho * a.chunks + lane];
    M = p.x;
    S = p.y;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) merge(M, S, __shfl_xor(M, off), __shfl_xor(S, off), a.c);
  return make_float2(M, S);
}

// Row of slot t of sequence i: slot r <= k is target row r, slot k+1+r
// draft row r.
__device__ __forceinline__ int64_t slot_row(const SampleArgs& a, int i, int t) {
  const int k = a.k;
  return t <= k ? static_cast<int64_t>(i) * (k + 1) + t
                : static_cast<int64_t>(a.B) * (k + 1) + static_cast<int64_t>(i) * k + (t - k - 1);
}

// Normalisers of all 2k+1 slots of sequence i into LDS, one wave per slot.
__device__ __forceinline__ void row_norms(const SampleArgs& a, int i, float* rowM, float* rowS) {
  const int wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int t = wave; t < 2 * a.k + 1; t += nw) {
    const float2 n = row_norm(a, slot_row(a, i, t));
    if ((threadIdx.x & 63) == 0) {
      rowM[t] = n.x;
      rowS[t] = n.y;
    }
  }
}

// Acceptance tests of sequence i, one lane of wave 0 per draft: draft r is
// accepted iff u_r * q_r(x_r) < p_r(x_r).  draft_logit_pair loads the two
// logits at x_r (issued before the normalisers are known); accepted_count
// returns (to wave 0) the first rejected slot, k if none.
struct DraftLogits {
  float lt, ld, u;
  bool valid;
};

template <int DT>
__device__ __forceinline__ DraftLogits draft_logit_pair(const SampleArgs& a, int i, bool flag) {
  constexpr int eb = DT == 0 ? 4 : 2;
  const int k = a.k;
  const int64_t V = a.V;
  DraftLogits d{0.0f, 0.0f, 0.0f, false};
  const int r = threadIdx.x;
  if (r < k) {
    float u = a.u_accept[static_cast<int64_t>(i) * k + r];
    if (!(u >= 0.0f && u < 1.0f)) {
      if (flag && a.dev_status) atomicOr(a.dev_status, kBadUniform);
      u = u >= 1.0f ? 0.99999994f : 0.0f;
    }
    d.u = u;
    const int32_t x = a.draft[static_cast<int64_t>(i) * k + r];
    if (x >= 0 && x < V) {
      d.valid = true;
      d.lt = widen<DT>(a.logits + (static_cast<int64_t>(i) * (k + 1) + r) * V * eb, x);
      d.ld = widen<DT>(a.draft_logits + (static_cast<int64_t>(i) * k + r) * V * eb, x);
    }
  }
  return d;
}

__device__ __forceinline__ int accepted_count(const SampleArgs& a, const DraftLogits& d, const float* rowM,
                                              const float* rowS) {
  const int k = a.k;
  const int r = threadIdx.x;
  bool reject = false;
  if (r < k) {
    float px = 0.0f, qx = 0.0f;
    if (d.valid) {
      px = ex2((d.lt - rowM[r]) * a.c) / rowS[r];
      qx = ex2((d.ld - rowM[k + 1 + r]) * a.c) / rowS[k + 1 + r];
    }
    reject = !(d.u * qx < px);
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
  // n = (target max, 1 / target sum, draft max, 1 / draft sum) of slot j
  __device__ void init(const SampleArgs& a, int i, int j, float4 n) {
    constexpr int eb = DT == 0 ? 4 : 2;
    const int k = a.k;
    residual = j < k;
    trow = a.logits + (static_cast<int64_t>(i) * (k + 1) + j) * a.V * eb;
    drow = residual ? a.draft_logits + (static_cast<int64_t>(i) * k + j) * a.V * eb : trow;
    tM = n.x;
    tinv = n.y;
    dM = residual ? n.z : 0.0f;
    dinv = residual ? n.w : 0.0f;
    ta = row_aligned(trow, eb);
    da = row_aligned(drow, eb);
  }
  // residual weights (0 when there is no residual) and target weights of a group
  __device__ __forceinline__ void weights(int64_t g, int64_t end, float c, float (&wr)[kGroup],
                                          float (&wp)[kGroup]) const {
    float xt[kGroup];
    load_group<DT>(trow, g, end, ta, xt);
#pragma unroll
    for (int e = 0; e < kGroup; ++e) wp[e] = ex2((xt[e] - tM) * c);
    if (residual) {
      float xd[kGroup];
      load_group<DT>(drow, g, end, da, xd);
#pragma unroll
      for (int e = 0; e < kGroup; ++e) wr[e] = fmaxf(wp[e] * tinv - ex2((xd[e] - dM) * c) * dinv, 0.0f);
    } else {
#pragma unroll
      for (int e = 0; e < kGroup; ++e) wr[e] = 0.0f;
    }
  }
};

constexpr int kAcceptThreads = 256;
constexpr int kMassThreads = 256;               // kMassThreads * kGroup == kTile: one tile per iteration
constexpr int kPickThreads = 256;
static_assert(kMassThreads * kGroup == kTile && kPickThreads * kGroup == kTile, "a tile is one group per thread");
constexpr int kMaxTiles = 64;                   // tiles per chunk (V <= 64 * 64 * kTile)
constexpr int64_t kMassTarget = 2048;           // mass workgroups the chunking aims for

// One workgroup per sequence: the normalisers of its 2k+1 rows (one wave per
// row), the acceptance tests (wave 0), then n_acc and the normalisers of the
// rows the sequence samples from.
template <int DT>
__global__ __launch_bounds__(kAcceptThreads) void sample_accept_kernel(SampleArgs a) {
  __shared__ float rowM[2 * (64 + 1)], rowS[2 * (64 + 1)];
  const int i = blockIdx.x;
  const int k = a.k;
  DraftLogits dl{0.0f, 0.0f, 0.0f, false};
  if (threadIdx.x < 64) dl = draft_logit_pair<DT>(a, i, true);
  row_norms(a, i, rowM, rowS);
  __syncthreads();
  if (threadIdx.x < 64) {
    const int j = accepted_count(a, dl, rowM, rowS);
    if (threadIdx.x == 0) {
      a.n_acc[i] = j;
      a.norms[i] = make_float4(rowM[j], 1.0f / rowS[j], j < k ? rowM[k + 1 + j] : 0.0f,
                               j < k ? 1.0f / rowS[k + 1 + j] : 0.0f);
    }
  }
}

// One workgroup per (sequence, chunk): tile by tile, the total residual and
// target weight of each kTile logits of the chunk, and the last index of
// positive weight of each over the chunk.
template <int DT>
__global__ __launch_bounds__(kMassThreads) void sample_mass_kernel(SampleArgs a) {
  __shared__ float2 tsum[kMaxTiles][kMassThreads / 64];
  __shared__ int32_t redi[2][kMassThreads / 64];
  const int i = static_cast<int>(blockIdx.x / a.mchunks);
  const int64_t chunk = blockIdx.x - static_cast<int64_t>(i) * a.mchunks;
  SampleRows<DT> rows;
  rows.init(a, i, a.n_acc[i], a.norms[i]);
  const int64_t beg = chunk * a.mchunk_elems;
  int64_t end = beg + a.mchunk_elems;
  if (end > a.V) end = a.V;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int32_t lr = -1, lp = -1;
  int t = 0;
  for (int64_t g = beg / kGroup + threadIdx.x; (g - threadIdx.x) * kGroup < end; g += kMassThreads, ++t) {
    float sr = 0.0f, sp = 0.0f;
    if (g * kGroup < end) {
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
    }
    if (lane == 0) tsum[t][wave] = make_float2(sr, sp);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t o1 = __shfl_xor(lr, off), o2 = __shfl_xor(lp, off);
    lr = o1 > lr ? o1 : lr;
    lp = o2 > lp ? o2 : lp;
  }
  if (lane == 0) {
    redi[0][wave] = lr;
    redi[1][wave] = lp;
  }
  __syncthreads();
  // tile totals in wave order (fixed), one thread per tile
  for (int tt = threadIdx.x; tt < t; tt += kMassThreads) {
    float r = 0.0f, q = 0.0f;
#pragma unroll
    for (int w = 0; w < kMassThreads / 64; ++w) {
      r += tsum[tt][w].x;
      q += tsum[tt][w].y;
    }
    a.mass[(static_cast<int64_t>(blockIdx.x)) * a.tiles + tt] = make_float2(r, q);
  }
  for (int tt = t + threadIdx.x; tt < a.tiles; tt += kMassThreads)
    a.mass[(static_cast<int64_t>(blockIdx.x)) * a.tiles + tt] = make_float2(0.0f, 0.0f);
  if (threadIdx.x == 0) {
    int32_t mr = -1, mp = -1;
#pragma unroll
    for (int w = 0; w < kMassThreads / 64; ++w) {
      mr = redi[0][w] > mr ? redi[0][w] : mr;
      mp = redi[1][w] > mp ? redi[1][w] : mp;
    }
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

// Wave 0: inclusive prefix, from `base`, of n <= 64 values (one per lane;
// lanes beyond n hold 0); returns the first lane whose running total exceeds
// `target` and, in *excl, the running total before it.  Where rounding leaves
// no such lane, the last lane of positive value is returned instead (-1 if
// every value is 0).
__device__ __forceinline__ int first_crossing(float v, int n, float base, float target, float* excl) {
  const int c = threadIdx.x;
  const bool positive = c < n && v > 0.0f;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float o = __shfl_up(v, off);
    if (c >= off) v += o;
  }
  const float incl = base + v;
  const float prev = __shfl_up(incl, 1);
  const unsigned long long hit = __ballot(c < n && incl > target);
  const unsigned long long pos = __ballot(positive);
  const int cs = hit ? __builtin_ctzll(hit) : (pos ? 63 - __builtin_clzll(pos) : -1);
  *excl = __shfl(c == 0 ? base : prev, cs < 0 ? 0 : cs);
  return cs;
}

// New width and paddings (Eq. (1), Eq. (2)) from the accepted counts, by one
// workgroup of kPickThreads.
__device__ void width_and_pads(const SampleArgs& a, int32_t* red) {
  const int32_t L = a.W_in - (a.k + 1);
  int32_t local = 0;
  for (int i = threadIdx.x; i < a.B; i += kPickThreads) {
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
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = local;
  __syncthreads();
  int32_t w = red[0];
#pragma unroll
  for (int q = 1; q < kPickThreads / 64; ++q) w = red[q] > w ? red[q] : w;
  for (int i = threadIdx.x; i < a.B; i += kPickThreads) {
    const int32_t p = a.pad_in[i];
    a.pad_out[i] = (p >= 0 && p <= L) ? w - ((L - p) + a.n_acc[i] + 1) : -1;
  }
  if (threadIdx.x == 0) a.w_new[0] = w;
}

// One workgroup per sequence: inversion with u_sample, coarse to fine: the
// chunk totals (wave 0, at most 64 chunks), the tile totals of the crossing
// chunk (wave 0), then one block-wide scan of the crossing tile.  A residual
// with no mass falls back to p_j; where rounding leaves no crossing, the last
// index of positive weight seen is taken.  Workgroup 0 also writes the new
// width and paddings.
template <int DT>
__global__ __launch_bounds__(kPickThreads) void sample_pick_kernel(SampleArgs a) {
  __shared__ float red[kPickThreads / 64];
  __shared__ int32_t redl[kPickThreads / 64];
  __shared__ int32_t s_tile, s_first, s_pick, s_fallback, s_use_res;
  __shared__ float s_excl, s_target;
  const int i = blockIdx.x;
  const int k = a.k;
  const int j = a.n_acc[i];
  if (blockIdx.x == 0) width_and_pads(a, redl);
  if (threadIdx.x < 64) {
    const int c = threadIdx.x;
    const int64_t wg0 = static_cast<int64_t>(i) * a.mchunks;  // mass workgroups of this sequence
    float cr = 0.0f, cp = 0.0f;
    if (c < a.mchunks)
      for (int tt = 0; tt < a.tiles; ++tt) {
        const float2 m = a.mass[(wg0 + c) * a.tiles + tt];
        cr += m.x;
        cp += m.y;
      }
    const int2 l = c < a.mchunks ? a.last[wg0 + c] : make_int2(-1, -1);
    float rtot = cr;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) rtot += __shfl_xor(rtot, off);
    const bool use_res = j < k && rtot > 0.0f;
    float v = use_res ? cr : cp;
    int32_t lastpos = use_res ? l.x : l.y;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(lastpos, off);
      lastpos = o > lastpos ? o : lastpos;
    }
    float total = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_up(total, off);
      if (c >= off) total += o;
    }
    total = __shfl(total, 63);
    float us = a.u_sample[i];
    if (!(us >= 0.0f && us < 1.0f)) {
      if (c == 0 && a.dev_status) atomicOr(a.dev_status, kBadUniform);
      us = us >= 1.0f ? 0.99999994f : 0.0f;
    }
    const float target = us * total;
    float excl_chunk = 0.0f;
    const int cs = first_crossing(v, a.mchunks, 0.0f, target, &excl_chunk);
    int ts = -1;
    float excl_tile = 0.0f;
    if (cs >= 0) {
      const float2 m = c < a.tiles ? a.mass[(wg0 + cs) * a.tiles + c] : make_float2(0.0f, 0.0f);
      ts = first_crossing(use_res ? m.x : m.y, a.tiles, excl_chunk, target, &excl_tile);
    }
    if (c == 0) {
      s_tile = cs >= 0 && ts >= 0 ? cs * a.tiles + ts : -1;   // tile index within the row
      s_excl = excl_tile;
      s_fallback = lastpos;
      s_use_res = use_res ? 1 : 0;
      s_target = target;
      s_pick = -1;
    }
  }
  __syncthreads();
  const int tile = s_tile;
  if (tile >= 0) {
    SampleRows<DT> rows;
    rows.init(a, i, j, a.norms[i]);
    const bool use_res = s_use_res != 0;
    const float target = s_target;
    const int cs = tile / a.tiles, ts = tile - cs * a.tiles;
    const int64_t cbeg = static_cast<int64_t>(cs) * a.mchunk_elems;
    int64_t cend = cbeg + a.mchunk_elems;
    if (cend > a.V) cend = a.V;
    const int64_t g = (cbeg + static_cast<int64_t>(ts) * kTile) / kGroup + threadIdx.x;
    float w[kGroup] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (g * kGroup < cend) {
      float wr[kGroup], wp[kGroup];
      rows.weights(g, cend, a.c, wr, wp);
#pragma unroll
      for (int e = 0; e < kGroup; ++e) w[e] = use_res ? wr[e] : wp[e];
    }
    float gs = 0.0f;
    int32_t lastg = -1;
#pragma unroll
    for (int e = 0; e < kGroup; ++e) {
      gs += w[e];
      if (w[e] > 0.0f) lastg = static_cast<int32_t>(g * kGroup + e);
    }
    float tt = 0.0f;
    const float incl = s_excl + block_inclusive_scan<kPickThreads>(gs, red, &tt);
    if (threadIdx.x == 0) s_first = 0x7FFFFFFF;
    __syncthreads();
    if (incl > target) atomicMin(&s_first, static_cast<int32_t>(threadIdx.x));
    __syncthreads();
    if (static_cast<int32_t>(threadIdx.x) == s_first) {
      float c = incl - gs;
      int32_t pick = -1;
#pragma unroll
      for (int e = 0; e < kGroup; ++e) {
        c += w[e];
        if (pick < 0 && c > target && w[e] > 0.0f) pick = static_cast<int32_t>(g * kGroup + e);
      }
      s_pick = pick >= 0 ? pick : lastg;
    }
    // no crossing inside the tile (rounding): the tile's last positive weight
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(lastg, off);
      lastg = o > lastg ? o : lastg;
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) redl[threadIdx.x >> 6] = lastg;
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
  if (static_cast<int>(threadIdx.x) <= k) {
    const int r = static_cast<int>(threadIdx.x);
    a.tokens[static_cast<int64_t>(i) * (k + 1) + r] =
        r < j ? a.draft[static_cast<int64_t>(i) * k + r] : (r == j ? x_out : -1);
  }
  if (threadIdx.x == 0 && a.bonus) a.bonus[i] = x_out;
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

int64_t sample_mass_chunk_elems(int64_t B, int64_t V) {
  // at most 64 chunks per row (one lane each in the pick kernel), at least
  // one tile each, and about kMassTarget workgroups in all: 8 of 256 threads
  // per CU, so the whole grid is resident at once (at B = 64, V = 151936,
  // 64 chunks per row took two rounds of workgroups: 13.4 us against 11.5)
  int64_t c = (V + 63) / 64;
  int64_t t = (B * V + kMassTarget - 1) / kMassTarget;
  if (t > kMaxTiles * kTile) t = kMaxTiles * kTile;   // at most kMaxTiles tiles a chunk
  if (t > c) c = t;
  c = ((c + kGroup - 1) / kGroup) * kGroup;
  if (c < kTile) c = kTile;
  if (c > V) c = V;
  return c;
}

static hipError_t sample_args(const SampleLaunch& p, SampleArgs& a) {
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
  a.mchunk_elems = sample_mass_chunk_elems(p.B, p.V);
  a.mchunks = static_cast<int32_t>((p.V + a.mchunk_elems - 1) / a.mchunk_elems);
  a.tiles = static_cast<int32_t>((a.mchunk_elems + kTile - 1) / kTile);
  if (a.tiles > kMaxTiles || a.mchunks > 64) return hipErrorInvalidValue;
  char* ws = static_cast<char*>(p.workspace) + kWsHeaderBytes;
  a.norms = reinterpret_cast<float4*>(ws);
  ws += static_cast<int64_t>(p.B) * 16;
  a.partial = reinterpret_cast<float2*>(ws);
  a.last = reinterpret_cast<int2*>(ws + rows * a.chunks * 8);
  a.mass = reinterpret_cast<float2*>(ws + (rows * a.chunks + static_cast<int64_t>(p.B) * a.mchunks) * 8);
  return hipSuccess;
}

hipError_t launch_sample_stats(const SampleLaunch& p, hipStream_t stream) {
  SampleArgs a{};
  const hipError_t r = sample_args(p, a);
  if (r != hipSuccess) return r;
  const int64_t rows = static_cast<int64_t>(p.B) * (2 * p.k + 1);
  const dim3 grid(static_cast<uint32_t>(rows * a.chunks));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_stats_kernel<0>, grid, dim3(kStatsThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_stats_kernel<1>, grid, dim3(kStatsThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_stats_kernel<2>, grid, dim3(kStatsThreads), 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_sample_finish(const SampleLaunch& p, hipStream_t stream) {
  SampleArgs a{};
  hipError_t e = sample_args(p, a);
  if (e != hipSuccess) return e;
  const dim3 seqs(static_cast<uint32_t>(p.B));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_accept_kernel<0>, seqs, dim3(kAcceptThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_accept_kernel<1>, seqs, dim3(kAcceptThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_accept_kernel<2>, seqs, dim3(kAcceptThreads), 0, stream, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 mgrid(static_cast<uint32_t>(static_cast<int64_t>(p.B) * a.mchunks));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_mass_kernel<0>, mgrid, dim3(kMassThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_mass_kernel<1>, mgrid, dim3(kMassThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_mass_kernel<2>, mgrid, dim3(kMassThreads), 0, stream, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_pick_kernel<0>, seqs, dim3(kPickThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_pick_kernel<1>, seqs, dim3(kPickThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_pick_kernel<2>, seqs, dim3(kPickThreads), 0, stream, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_verify_sample(const SampleLaunch& p, hipStream_t stream) {
  const hipError_t e = launch_sample_stats(p, stream);
  return e != hipSuccess ? e : launch_sample_finish(p, stream);
}

}  // namespace specdec
