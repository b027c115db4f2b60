// HIP kernels of the two rollback strategies of arXiv 2510.22876, Section 2
// ("Family A: contiguous layout", "Family B: variable-length layout"), on
// MI355X (gfx950, wave64).
//
//   rollback_kernel     Family A: one workgroup truncates every row to the
//                       batch-minimum accepted count m and applies Eq. (1) /
//                       Eq. (2) with a_i = m + 1 (all offsets equal: the cache
//                       realignment that follows moves nothing in place).
//   varlen_offsets      Family B: one workgroup computes each sequence's kept
//                       length (its rows minus its rejected window entries)
//                       and their running sum, the new cumulative offsets.
//   varlen_compact      Family B: the flat [T][H][D] cache of every (layer,
//                       K/V) is compacted into a second buffer, one sequence's
//                       kept rows per span, in the split-piece layout of the
//                       other out-of-place copies; extra workgroups write the
//                       position ids (I2: each row's index in its sequence).
#include "posmask.h"
#include "span_copy.h"
#include "specdec_internal.h"

namespace specdec {
namespace {

constexpr uint32_t kBadPadIn = 0x1u, kBadAccept = 0x2u, kBadWidth = 0x4u;
constexpr int kOneBlock = 1024;

__device__ __forceinline__ int32_t block_min_i32(int32_t v, int32_t* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t o = __shfl_xor(v, off);
    v = o < v ? o : v;
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  int32_t m = red[0];
#pragma unroll
  for (int q = 1; q < kOneBlock / 64; ++q) m = red[q] < m ? red[q] : m;
  return m;
}

__device__ __forceinline__ int32_t block_max_i32(int32_t v, int32_t* red) {
  return -block_min_i32(-v, red);
}

struct RollbackArgs {
  const int32_t* tokens;
  const int32_t* n_acc_in;
  const int32_t* pad_in;
  int32_t B, k, W_in;
  int32_t* n_acc_out;   // may equal n_acc_in
  int32_t* bonus_out;
  int32_t* pad_out;     // may equal pad_in
  int32_t* w_new;
  uint32_t* dev_status;
};

__global__ __launch_bounds__(kOneBlock) void rollback_kernel(RollbackArgs a) {
  __shared__ int32_t red[kOneBlock / 64];
  const int32_t L = a.W_in - (a.k + 1);
  // every input is read before any output is written (outputs may alias them)
  int32_t m = a.k;
  for (int i = threadIdx.x; i < a.B; i += kOneBlock) {
    const int32_t p = a.pad_in[i], n = a.n_acc_in[i];
    uint32_t err = 0u;
    if (p < 0 || p > L) err |= kBadPadIn;
    if (n < 0 || n > a.k) err |= kBadAccept;
    if (err) {
      if (a.dev_status) atomicOr(a.dev_status, err);
    } else {
      m = n < m ? n : m;
    }
  }
  m = block_min_i32(m, red);
  int32_t w = 0;
  for (int i = threadIdx.x; i < a.B; i += kOneBlock) {
    const int32_t p = a.pad_in[i], n = a.n_acc_in[i];
    if (p >= 0 && p <= L && n >= 0 && n <= a.k) {
      const int32_t len = (L - p) + m + 1;               // Eq. (1) with a_i = m + 1
      w = len > w ? len : w;
    }
  }
  w = block_max_i32(w, red);
  // each thread writes only the rows it reads here, after the block-wide
  // reductions: outputs may alias the inputs
  for (int i = threadIdx.x; i < a.B; i += kOneBlock) {
    const int32_t p = a.pad_in[i], n = a.n_acc_in[i];
    const bool ok = p >= 0 && p <= L && n >= 0 && n <= a.k;
    a.bonus_out[i] = ok ? a.tokens[static_cast<int64_t>(i) * (a.k + 1) + m] : -1;
    // Eq. (2): delta = (w - L) - (m + 1), the same for every row
    a.pad_out[i] = ok ? p + ((w - L) - (m + 1)) : -1;
    a.n_acc_out[i] = ok ? m : n;
  }
  if (threadIdx.x == 0) a.w_new[0] = w;
}

// ---- Family B ------------------------------------------------------------------

constexpr int kTpb = 64;
constexpr int kPieces = 2;
constexpr int kSplit = 512;
constexpr int kNt = 3;

struct VarlenArgs {
  const u32x4* src;
  u32x4* dst;
  int64_t src_slab_vecs, dst_slab_vecs;  // T_cap * H * D / 8 per (layer, K/V)
  int64_t row_vecs;                      // H * D / 8: one token row of the flat buffer
  int64_t src_T, dst_T;
  const int32_t* cu_in;
  const int32_t* n_acc;
  int32_t* cu_out;
  int64_t* pos;
  int32_t B, k, max_len;
  uint32_t* dev_status;
  uint32_t chunks;        // workgroups per span
  uint32_t span_base;
  uint32_t pos_blocks;    // position-id workgroups (first launch only)
  uint32_t pos_col_blocks;
};

// Kept lengths and their running sum (one workgroup, B in stripes of 1024).
__global__ __launch_bounds__(kOneBlock) void varlen_offsets_kernel(VarlenArgs a) {
  __shared__ int32_t wsum[kOneBlock / 64];
  __shared__ int32_t carry;
  if (threadIdx.x == 0) {
    carry = 0;
    a.cu_out[0] = 0;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int i0 = 0; i0 < a.B; i0 += kOneBlock) {
    const int i = i0 + threadIdx.x;
    int32_t keep = 0;
    if (i < a.B) {
      const int64_t b = a.cu_in[i], e = a.cu_in[i + 1];
      const int32_t n = a.n_acc[i];
      uint32_t err = 0u;
      if (b < 0 || e < b || e > a.src_T || e - b < a.k + 1 || e - b > a.max_len) err |= kBadWidth;
      if (n < 0 || n > a.k) err |= kBadAccept;
      if (err) {
        if (a.dev_status) atomicOr(a.dev_status, err);
      } else {
        keep = static_cast<int32_t>(e - b) - (a.k - n);
      }
    }
    // inclusive scan of keep over the stripe
    int32_t v = keep;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t o = __shfl_up(v, off);
      if (lane >= off) v += o;
    }
    if (lane == 63) wsum[wave] = v;
    __syncthreads();
    int32_t before = carry;
#pragma unroll
    for (int q = 0; q < kOneBlock / 64; ++q) before += q < wave ? wsum[q] : 0;
    if (i < a.B) a.cu_out[i + 1] = before + v;
    __syncthreads();
    if (threadIdx.x == kOneBlock - 1) carry = before + v;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kTpb) void varlen_compact_kernel(VarlenArgs a) {
  uint32_t b = blockIdx.x;
  if (b < a.pos_blocks) {
    // position ids of one sequence's kept rows: 4*kTpb rows per workgroup
    const uint32_t i = b / a.pos_col_blocks;
    const uint32_t cb = b - i * a.pos_col_blocks;
    const int64_t o = load_invariant(a.cu_out + i);
    const int64_t keep = load_invariant(a.cu_out + i + 1) - o;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t t = static_cast<int64_t>(cb) * (4 * kTpb) + q * kTpb + threadIdx.x;
      if (t < keep) a.pos[o + t] = t;
    }
    return;
  }
  b -= a.pos_blocks;
  const uint32_t rel = b / a.chunks;
  const uint32_t sub = b - rel * a.chunks;
  const uint32_t span = a.span_base + rel;                // (layer*2 + kv) * B + i
  const uint32_t lk = span / static_cast<uint32_t>(a.B);
  const int i = static_cast<int>(span - lk * static_cast<uint32_t>(a.B));
  const int64_t o = load_invariant(a.cu_out + i);
  const int64_t keep = load_invariant(a.cu_out + i + 1) - o;   // 0 for a skipped sequence
  const int64_t from = load_invariant(a.cu_in + i);
  const int64_t total = keep * a.row_vecs;
  u32x4* d = a.dst + static_cast<int64_t>(lk) * a.dst_slab_vecs + o * a.row_vecs;
  const int64_t base = split_base<kPieces, kTpb, kSplit>(sub) - split_misalign<kPieces, kSplit>(d);
  if (base >= total) return;
  split_pieces<kPieces, kTpb, kSplit, kNt>(a.src + static_cast<int64_t>(lk) * a.src_slab_vecs + from * a.row_vecs, d,
                                           base, total, 0, 0);
}

}  // namespace

hipError_t launch_rollback(const RollbackLaunch& p, hipStream_t stream) {
  RollbackArgs a{p.tokens, p.n_acc_in, p.pad_in, p.B, p.k, p.W_in, p.n_acc_out, p.bonus_out, p.pad_out, p.w_new,
                 p.dev_status};
  hipLaunchKernelGGL(rollback_kernel, dim3(1), dim3(kOneBlock), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_varlen_rollback(const VarlenLaunch& p, hipStream_t stream) {
  VarlenArgs a{};
  a.src = static_cast<const u32x4*>(p.src);
  a.dst = static_cast<u32x4*>(p.dst);
  a.row_vecs = static_cast<int64_t>(p.H) * p.D / 8;
  a.src_slab_vecs = p.src_T * a.row_vecs;
  a.dst_slab_vecs = p.dst_T * a.row_vecs;
  a.src_T = p.src_T;
  a.dst_T = p.dst_T;
  a.cu_in = p.cu_in;
  a.n_acc = p.n_acc;
  a.cu_out = p.cu_out;
  a.pos = p.pos;
  a.B = p.B;
  a.k = p.k;
  a.max_len = p.max_len;
  a.dev_status = p.dev_status;
  hipLaunchKernelGGL(varlen_offsets_kernel, dim3(1), dim3(kOneBlock), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  a.pos_col_blocks = static_cast<uint32_t>((static_cast<int64_t>(p.max_len) + 4 * kTpb - 1) / (4 * kTpb));
  const int64_t pos_blocks = p.pos ? static_cast<int64_t>(a.pos_col_blocks) * p.B : 0;
  const int64_t nspans = static_cast<int64_t>(p.L) * 2 * p.B;
  // every span may start anywhere: room for the extra group of the aligned tiling
  const int64_t chunks = split_blocks<kPieces, kTpb, kSplit>(static_cast<int64_t>(p.max_len) * a.row_vecs, true);
  a.chunks = static_cast<uint32_t>(chunks);
  const int64_t per_launch = (max_launch_items() / kTpb - pos_blocks) / chunks;
  if (per_launch < 1) return hipErrorInvalidConfiguration;
  for (int64_t s0 = 0; s0 == 0 || s0 < nspans; s0 += per_launch) {
    const int64_t ns = nspans - s0 < per_launch ? nspans - s0 : per_launch;
    const bool first = s0 == 0;
    a.span_base = static_cast<uint32_t>(s0);
    a.pos_blocks = first ? static_cast<uint32_t>(pos_blocks) : 0u;
    const int64_t blocks = ns * chunks + (first ? pos_blocks : 0);
    if (blocks > 0) {
      hipLaunchKernelGGL(varlen_compact_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTpb), 0, stream, a);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if (ns <= 0) break;
  }
  return hipSuccess;
}

}  // namespace specdec
