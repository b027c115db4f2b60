// HIP kernels of stochastic (temperature T > 0) verification on MI355X
// (gfx950, wave64): speculative sampling over a batch, the T > 0 counterpart of
// greedy BatchVerify (arXiv 2510.22876, Algorithm 3; the target-distribution
// requirement of output equivalence at T > 0).
//
//   sample_stats    every target and draft logit row, split over workgroups:
//                   the row maximum and the sum of exp((x - max) / T) of each
//                   chunk (online: a thread rescales its sum when its maximum
//                   grows), stored per chunk.
//   sample_decide   one workgroup per sequence: combines the chunk sums into
//                   p_r = softmax(target_r / T) and q_r = softmax(draft_r / T)
//                   normalisers, accepts draft r iff u_r * q_r(x_r) < p_r(x_r)
//                   (wave 0, one lane per draft, first rejection by ballot),
//                   then samples the correction from max(0, p_r - q_r) (or the
//                   bonus from p_k) by inversion: one pass for the total mass,
//                   then a tiled prefix scan that stops at the tile where the
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
constexpr int kDecideThreads = 1024;
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

// Block-wide sum (kDecideThreads threads); every thread gets the total.
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float t = 0.0f;
#pragma unroll
  for (int q = 0; q < kDecideThreads / 64; ++q) t += red[q];
  return t;
}

// Inclusive prefix sum over the block in thread order; *total gets the sum.
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
  for (int q = 0; q < kDecideThreads / 64; ++q) {
    const float r = red[q];
    before += q < wave ? r : 0.0f;
    all += r;
  }
  *total = all;
  return before + v;
}

template <int DT>
__global__ __launch_bounds__(kDecideThreads) void sample_decide_kernel(SampleArgs a) {
  constexpr int eb = DT == 0 ? 4 : 2;
  __shared__ float rowM[2 * (64 + 1)], rowS[2 * (64 + 1)];
  __shared__ float red[kDecideThreads / 64];
  __shared__ int32_t redi[kDecideThreads / 64];
  __shared__ int32_t s_nacc, s_first, s_pick;
  const int i = blockIdx.x;
  const int k = a.k;
  const int64_t V = a.V;
  const int64_t nt = static_cast<int64_t>(a.B) * (k + 1);
  // (1) normalisers of the sequence's 2k+1 rows: slot r <= k target row r,
  //     slot k+1+r draft row r
  for (int t = threadIdx.x; t < 2 * k + 1; t += kDecideThreads) {
    const int64_t rho = t <= k ? static_cast<int64_t>(i) * (k + 1) + t : nt + static_cast<int64_t>(i) * k + (t - k - 1);
    const float2* p = a.partial + rho * a.chunks;
    float M = p[0].x, S = p[0].y;
    for (int q = 1; q < a.chunks; ++q) merge(M, S, p[q].x, p[q].y, a.c);
    rowM[t] = M;
    rowS[t] = S;
  }
  __syncthreads();
  // (2) acceptance tests, one lane of wave 0 per draft
  if (threadIdx.x < 64) {
    bool reject = false;
    const int r = threadIdx.x;
    if (r < k) {
      float u = a.u_accept[static_cast<int64_t>(i) * k + r];
      if (!(u >= 0.0f && u < 1.0f)) {
        if (a.dev_status) atomicOr(a.dev_status, kBadUniform);
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
    if (threadIdx.x == 0) s_nacc = rej ? __builtin_ctzll(rej) : k;
  }
  __syncthreads();
  const int j = s_nacc;
  // (3) sampling by inversion over the weights of slot j
  const bool residual = j < k;
  const char* trow = a.logits + (static_cast<int64_t>(i) * (k + 1) + j) * V * eb;
  const char* drow = residual ? a.draft_logits + (static_cast<int64_t>(i) * k + j) * V * eb : trow;
  const float tM = rowM[j], tinv = 1.0f / rowS[j];
  const float dM = residual ? rowM[k + 1 + j] : 0.0f, dinv = residual ? 1.0f / rowS[k + 1 + j] : 0.0f;
  const bool ta = row_aligned(trow, eb), da = row_aligned(drow, eb);
  float us = a.u_sample[i];
  if (!(us >= 0.0f && us < 1.0f)) {
    if (threadIdx.x == 0 && a.dev_status) atomicOr(a.dev_status, kBadUniform);
    us = us >= 1.0f ? 0.99999994f : 0.0f;
  }
  const int64_t ngroups = (V + kGroup - 1) / kGroup;
  // weights of one group: residual max(0, p - q), or p (unnormalised: e / 1)
  auto weights = [&](int64_t g, bool use_residual, float (&w)[kGroup]) {
    float xt[kGroup];
    load_group<DT>(trow, g, V, ta, xt);
    if (use_residual) {
      float xd[kGroup];
      load_group<DT>(drow, g, V, da, xd);
#pragma unroll
      for (int e = 0; e < kGroup; ++e)
        w[e] = fmaxf(exp2f((xt[e] - tM) * a.c) * tinv - exp2f((xd[e] - dM) * a.c) * dinv, 0.0f);
    } else {
#pragma unroll
      for (int e = 0; e < kGroup; ++e) w[e] = exp2f((xt[e] - tM) * a.c);
    }
  };
  // pass 1: total mass (and the last index of positive weight, the fallback)
  bool use_residual = residual;
  float total = 0.0f;
  int32_t last = -1;
  for (int pass = 0; pass < 2; ++pass) {
    float part = 0.0f;
    int32_t lp = -1;
    for (int64_t g = threadIdx.x; g < ngroups; g += kDecideThreads) {
      float w[kGroup];
      weights(g, use_residual, w);
#pragma unroll
      for (int e = 0; e < kGroup; ++e) {
        part += w[e];
        if (w[e] > 0.0f) lp = static_cast<int32_t>(g * kGroup + e);
      }
    }
    total = block_sum(part, red);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const int32_t o = __shfl_xor(lp, off);
      lp = o > lp ? o : lp;
    }
    if ((threadIdx.x & 63) == 0) redi[threadIdx.x >> 6] = lp;
    __syncthreads();
    last = -1;
#pragma unroll
    for (int q = 0; q < kDecideThreads / 64; ++q) {
      const int32_t o = redi[q];
      last = o > last ? o : last;
    }
    __syncthreads();
    // a residual with no mass falls back to p_j
    if (total > 0.0f || !use_residual) break;
    use_residual = false;
  }
  // pass 2: tiles of kDecideThreads groups in order; stop at the tile where
  // the running mass first exceeds the target.  The lowest thread whose
  // inclusive sum exceeds it (chosen with an LDS atomic, so the choice is
  // deterministic even where rounding makes the sums non-monotone) scans its
  // group; if rounding leaves no crossing inside the group it takes the
  // group's last positive weight.
  const float target = us * total;
  if (threadIdx.x == 0) s_pick = -1;
  float running = 0.0f;
  for (int64_t g0 = 0; g0 < ngroups; g0 += kDecideThreads) {
    const int64_t g = g0 + threadIdx.x;
    float w[kGroup] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (g < ngroups) weights(g, use_residual, w);
    float gs = 0.0f;
#pragma unroll
    for (int e = 0; e < kGroup; ++e) gs += w[e];
    float tile = 0.0f;
    const float incl = running + block_inclusive_scan(gs, red, &tile);
    if (threadIdx.x == 0) s_first = 0x7FFFFFFF;
    __syncthreads();
    if (incl > target) atomicMin(&s_first, static_cast<int32_t>(threadIdx.x));
    __syncthreads();
    const int32_t first = s_first;
    if (first != 0x7FFFFFFF) {
      if (static_cast<int32_t>(threadIdx.x) == first) {
        float c = incl - gs;
        int32_t pick = -1, lastpos = -1;
#pragma unroll
        for (int e = 0; e < kGroup; ++e) {
          c += w[e];
          if (pick < 0 && c > target && w[e] > 0.0f) pick = static_cast<int32_t>(g * kGroup + e);
          if (w[e] > 0.0f) lastpos = static_cast<int32_t>(g * kGroup + e);
        }
        s_pick = pick >= 0 ? pick : lastpos;
      }
      break;
    }
    running += tile;
  }
  __syncthreads();
  int32_t x_out = s_pick;
  if (x_out < 0 || x_out >= V) x_out = last;   // rounding left no crossing: the last positive weight
  if (threadIdx.x <= k) {
    const int r = threadIdx.x;
    a.tokens[static_cast<int64_t>(i) * (k + 1) + r] =
        r < j ? a.draft[static_cast<int64_t>(i) * k + r] : (r == j ? x_out : -1);
  }
  if (threadIdx.x == 0) {
    a.n_acc[i] = j;
    if (a.bonus) a.bonus[i] = x_out;
  }
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
  a.partial = reinterpret_cast<float2*>(static_cast<char*>(p.workspace) + kWsHeaderBytes);
  a.dev_status = p.dev_status;
  const int64_t rows = static_cast<int64_t>(p.B) * (2 * p.k + 1);
  a.chunk_elems = sample_chunk_elems(rows, p.V);
  a.chunks = static_cast<int32_t>((p.V + a.chunk_elems - 1) / a.chunk_elems);
  const dim3 grid(static_cast<uint32_t>(rows * a.chunks));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_stats_kernel<0>, grid, dim3(kStatsThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_stats_kernel<1>, grid, dim3(kStatsThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_stats_kernel<2>, grid, dim3(kStatsThreads), 0, stream, a); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 seqs(static_cast<uint32_t>(p.B));
  switch (p.dtype) {
    case 0: hipLaunchKernelGGL(sample_decide_kernel<0>, seqs, dim3(kDecideThreads), 0, stream, a); break;
    case 1: hipLaunchKernelGGL(sample_decide_kernel<1>, seqs, dim3(kDecideThreads), 0, stream, a); break;
    default: hipLaunchKernelGGL(sample_decide_kernel<2>, seqs, dim3(kDecideThreads), 0, stream, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_width_kernel, dim3(1), dim3(1024), 0, stream, a);
  return hipGetLastError();
}

}  // namespace specdec
