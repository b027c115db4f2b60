// HIP kernels of EXSpec's pool traffic (arXiv 2510.22876, Algorithm 2) on
// MI355X (gfx950, wave64).
//
//   gather_kernel     GetBatch: rows of the sequence pool, each stored unpadded
//                     in its own slot, become a batch left-padded to the
//                     longest row.  Same-length rows are a plain concatenation
//                     (every padding is zero); otherwise this is the
//                     unpad-repad fallback.  The token rows, the paddings and
//                     the position ids / mask of the new batch (invariant I2)
//                     are written by extra workgroups of the same launch.
//   writeback_*       Write-back: each row's cache, unpadded and cut after its
//                     accepted entries, returns to its slot (whole, or only the
//                     new entries); its slot's token list and length grow.
//
// Both are bandwidth-bound gathers of whole (layer, K/V, row, head) spans of
// D-contiguous bf16 with 16-byte loads and stores; no matrix cores.
#include "posmask.h"
#include "span_copy.h"
#include "specdec_internal.h"

namespace specdec {
namespace {

constexpr uint32_t kBadPadIn = 0x1u, kBadAccept = 0x2u, kBadSlot = 0x10u, kSlotLen = 0x20u;

// The gather and the whole-row write-back use the out-of-place realignment's
// split-piece layout (64-thread workgroups, two 1 KB pieces 8 KB apart,
// nontemporal loads and stores): the access pattern is the same.
constexpr int kTpb = 64;
constexpr int kPieces = 2;
constexpr int kSplit = 512;
constexpr int kNt = 3;

struct GatherArgs {
  const u32x4* pool;
  u32x4* batch;
  int64_t pool_span_vecs, batch_span_vecs;  // cap * D / 8
  int32_t vpc;                              // 16-byte vectors per column
  int32_t N, B, H, Lb, k;
  int64_t pool_cap;
  const int32_t* pool_tok;
  int64_t pool_tok_stride;
  const int32_t* lens;
  const int32_t* slots;
  int32_t* batch_tok;
  int64_t btok_stride;
  int32_t pad_id;
  int32_t* pads;
  int64_t* pos;
  uint8_t* mask;
  int64_t pm_cap;
  uint32_t* dev_status;
  uint32_t chunks;        // workgroups per span
  uint32_t misaligned;    // batch spans tiled from the group boundary below them
  uint32_t span_base;     // first span of this launch
  uint32_t pm_blocks;     // position-id / mask workgroups (first launch only)
  uint32_t pm_col_blocks;
  uint32_t tok_blocks;    // token-row workgroups (first launch only)
  uint32_t tok_col_blocks;
};

// Length of the row's slot, or -1 when the slot or its length is out of
// range.  Every workgroup of a row takes the same decision.
__device__ __forceinline__ int32_t gather_row_len(const GatherArgs& a, int row, int32_t* slot_out) {
  const int32_t s = load_invariant(a.slots + row);
  *slot_out = s;
  if (s < 0 || s >= a.N) return -1;
  const int32_t n = load_invariant(a.lens + s);
  if (n < 0 || n > a.Lb || n > a.pool_cap) return -1;
  if (a.batch_tok && static_cast<int64_t>(n) + 1 > a.pool_tok_stride) return -1;
  return n;
}

__global__ __launch_bounds__(kTpb) void gather_kernel(GatherArgs a) {
  uint32_t b = blockIdx.x;
  if (b < a.pm_blocks) {
    // position ids and mask of the new batch: pad = Lb - n, width Lb + k + 1
    const uint32_t row = b / a.pm_col_blocks;
    const uint32_t cb = b - row * a.pm_col_blocks;
    int32_t slot;
    const int32_t n = gather_row_len(a, static_cast<int>(row), &slot);
    if (n < 0) return;
    posmask_cols<kTpb>(cb, a.pos + static_cast<int64_t>(row) * a.pm_cap, a.mask + static_cast<int64_t>(row) * a.pm_cap,
                       static_cast<int64_t>(a.Lb) - n, static_cast<int64_t>(a.Lb) + a.k + 1);
    return;
  }
  b -= a.pm_blocks;
  if (b < a.tok_blocks) {
    // token row (Lb + 1 columns) and padding of one row
    const uint32_t row = b / a.tok_col_blocks;
    const uint32_t cb = b - row * a.tok_col_blocks;
    int32_t slot;
    const int32_t n = gather_row_len(a, static_cast<int>(row), &slot);
    if (cb == 0 && threadIdx.x == 0) {
      a.pads[row] = n < 0 ? -1 : a.Lb - n;
      if (n < 0 && a.dev_status) atomicOr(a.dev_status, kBadSlot);
    }
    if (n < 0 || !a.batch_tok) return;
    const int64_t p = static_cast<int64_t>(a.Lb) - n;
    const int32_t* src = a.pool_tok + static_cast<int64_t>(slot) * a.pool_tok_stride;
    int32_t* dst = a.batch_tok + static_cast<int64_t>(row) * a.btok_stride;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t j = static_cast<int64_t>(cb) * (4 * kTpb) + q * kTpb + threadIdx.x;
      if (j <= a.Lb) dst[j] = j < p ? a.pad_id : src[j - p];
    }
    return;
  }
  b -= a.tok_blocks;
  const uint32_t rel = b / a.chunks;
  const uint32_t sub = b - rel * a.chunks;
  const uint32_t span = a.span_base + rel;                 // batch span ((l*2+kv)*B + row)*H + h
  const uint32_t H = static_cast<uint32_t>(a.H), BH = static_cast<uint32_t>(a.B) * H;
  const uint32_t lk = span / BH;
  const uint32_t rh = span - lk * BH;
  const int row = static_cast<int>(rh / H);
  const uint32_t h = rh - static_cast<uint32_t>(row) * H;
  int32_t slot;
  const int32_t n = gather_row_len(a, row, &slot);
  if (n < 0) return;                                        // flagged by the row's token workgroup
  u32x4* dspan = a.batch + static_cast<int64_t>(span) * a.batch_span_vecs;
  const int64_t mis = a.misaligned ? split_misalign<kPieces, kSplit>(dspan) : 0;
  const int64_t base = split_base<kPieces, kTpb, kSplit>(sub) - mis;
  const int64_t vpc = a.vpc;
  const int64_t total = static_cast<int64_t>(a.Lb) * vpc;
  if (base >= total) return;
  const int64_t pad = (static_cast<int64_t>(a.Lb) - n) * vpc;
  const int64_t pool_span = (static_cast<int64_t>(lk) * a.N + slot) * a.H + h;
  split_pieces<kPieces, kTpb, kSplit, kNt>(a.pool + pool_span * a.pool_span_vecs, dspan, base, total, pad, pad);
}

struct WritebackArgs {
  const u32x4* batch;
  u32x4* pool;
  int64_t batch_span_vecs, pool_span_vecs;
  int32_t vpc;
  int32_t N, B, H, k, Lb;
  int64_t pool_cap;
  const int32_t* pads;
  const int32_t* tokens;
  const int32_t* n_acc;
  const int32_t* slots;
  int32_t* pool_tok;
  int64_t pool_tok_stride;
  int32_t* lens;
  int32_t* batch_tok;
  int64_t btok_stride;
  uint32_t* dev_status;
  uint32_t chunks;        // workgroups per span
  uint32_t misaligned;    // whole-row mode: pool spans tiled from the group boundary below them
  uint32_t span_base;
  uint32_t meta_blocks;   // one per row (first launch only)
};

struct RowBack {
  int32_t slot, pad, n, a;
};

// Geometry of a row's write-back; returns the error bits (0 = valid).
__device__ __forceinline__ uint32_t writeback_row(const WritebackArgs& a, int row, RowBack& g) {
  g.slot = load_invariant(a.slots + row);
  g.pad = load_invariant(a.pads + row);
  const int32_t na = load_invariant(a.n_acc + row);
  uint32_t err = 0u;
  if (g.slot < 0 || g.slot >= a.N) err |= kBadSlot;
  if (na < 0 || na > a.k) err |= kBadAccept;
  if (g.pad < 0 || g.pad > a.Lb) err |= kBadPadIn;
  if (err) return err;
  g.n = a.Lb - g.pad;
  g.a = na + 1;
  const int64_t grown = static_cast<int64_t>(g.n) + g.a;
  if (grown > a.pool_cap || grown + 1 > a.pool_tok_stride) return kBadSlot;
  return 0u;
}

// Token lists and lengths: one workgroup per row.  The slot's length is read
// and rewritten by this workgroup only (the cache workgroups never read it).
__device__ void writeback_meta(const WritebackArgs& a, int row) {
  RowBack g;
  const uint32_t err = writeback_row(a, row, g);
  if (err) {
    if (threadIdx.x == 0 && a.dev_status) atomicOr(a.dev_status, err);
    return;
  }
  const int32_t* tk = a.tokens + static_cast<int64_t>(row) * (a.k + 1);
  int32_t* trow = a.pool_tok + static_cast<int64_t>(g.slot) * a.pool_tok_stride;
  for (int r = threadIdx.x; r < g.a; r += kTpb) trow[g.n + 1 + r] = tk[r];
  if (a.batch_tok) {
    int32_t* brow = a.batch_tok + static_cast<int64_t>(row) * a.btok_stride;
    for (int r = threadIdx.x; r < g.a; r += kTpb) brow[a.Lb + 1 + r] = tk[r];
  }
  if (threadIdx.x == 0) {
    const int32_t before = a.lens[g.slot];
    if (before != g.n && a.dev_status) atomicOr(a.dev_status, kSlotLen);
    a.lens[g.slot] = g.n + g.a;
  }
}

__device__ __forceinline__ void span_of(const WritebackArgs& a, uint32_t span, int& row, int64_t& pool_span_of_slot_base,
                                        uint32_t& lk, uint32_t& h) {
  const uint32_t H = static_cast<uint32_t>(a.H), BH = static_cast<uint32_t>(a.B) * H;
  lk = span / BH;
  const uint32_t rh = span - lk * BH;
  row = static_cast<int>(rh / H);
  h = rh - static_cast<uint32_t>(row) * H;
  pool_span_of_slot_base = static_cast<int64_t>(lk) * a.N;
}

// Whole row: pool columns [0, n + a) of the slot receive batch columns
// [pad, Lb + a) of the row, in the split-piece layout.
__global__ __launch_bounds__(kTpb) void writeback_full_kernel(WritebackArgs a) {
  uint32_t b = blockIdx.x;
  if (b < a.meta_blocks) {
    writeback_meta(a, static_cast<int>(b));
    return;
  }
  b -= a.meta_blocks;
  const uint32_t rel = b / a.chunks;
  const uint32_t sub = b - rel * a.chunks;
  const uint32_t span = a.span_base + rel;
  int row;
  int64_t lkN;
  uint32_t lk, h;
  span_of(a, span, row, lkN, lk, h);
  RowBack g;
  if (writeback_row(a, row, g)) return;   // flagged by the row's meta workgroup
  const int64_t vpc = a.vpc;
  u32x4* dspan = a.pool + ((lkN + g.slot) * a.H + h) * a.pool_span_vecs;
  const int64_t mis = a.misaligned ? split_misalign<kPieces, kSplit>(dspan) : 0;
  const int64_t base = split_base<kPieces, kTpb, kSplit>(sub) - mis;
  const int64_t total = static_cast<int64_t>(g.n + g.a) * vpc;
  if (base >= total) return;
  split_pieces<kPieces, kTpb, kSplit, kNt>(a.batch + static_cast<int64_t>(span) * a.batch_span_vecs, dspan, base,
                                           total, 0, -static_cast<int64_t>(g.pad) * vpc);
}

// New entries only: pool columns [n, n + a) of the slot receive batch columns
// [Lb, Lb + a) of the row; one workgroup per span (at most k + 1 columns).
__global__ __launch_bounds__(kTpb) void writeback_append_kernel(WritebackArgs a) {
  uint32_t b = blockIdx.x;
  if (b < a.meta_blocks) {
    writeback_meta(a, static_cast<int>(b));
    return;
  }
  const uint32_t span = a.span_base + (b - a.meta_blocks);
  int row;
  int64_t lkN;
  uint32_t lk, h;
  span_of(a, span, row, lkN, lk, h);
  RowBack g;
  if (writeback_row(a, row, g)) return;
  const int64_t vpc = a.vpc;
  const int64_t pool_span = (lkN + g.slot) * a.H + h;
  const u32x4* s = a.batch + static_cast<int64_t>(span) * a.batch_span_vecs + static_cast<int64_t>(a.Lb) * vpc;
  u32x4* d = a.pool + pool_span * a.pool_span_vecs + static_cast<int64_t>(g.n) * vpc;
  const int64_t nv = static_cast<int64_t>(g.a) * vpc;
  const int64_t w = static_cast<int64_t>(wave_index()) * 64;
  const int lane = static_cast<int>(threadIdx.x & 63);
  for (int64_t u0 = 0; u0 < nv; u0 += kTpb)
    if (u0 + w + lane < nv) st16_at<true>(d + (u0 + w), static_cast<uint32_t>(lane), ld16<true>(s + (u0 + w + lane)));
}

}  // namespace

hipError_t launch_gather(const GatherLaunch& p, hipStream_t stream) {
  GatherArgs a{};
  a.pool = static_cast<const u32x4*>(p.pool);
  a.batch = static_cast<u32x4*>(p.batch);
  a.vpc = p.D / 8;
  a.pool_span_vecs = p.pool_cap * a.vpc;
  a.batch_span_vecs = p.batch_cap * a.vpc;
  a.N = p.N;
  a.B = p.B;
  a.H = p.H;
  a.Lb = p.Lb;
  a.k = p.k;
  a.pool_cap = p.pool_cap;
  a.pool_tok = p.pool_tok;
  a.pool_tok_stride = p.pool_tok_stride;
  a.lens = p.lens;
  a.slots = p.slots;
  a.batch_tok = p.batch_tok;
  a.btok_stride = p.btok_stride;
  a.pad_id = p.pad_id;
  a.pads = p.pads;
  a.pos = p.pos;
  a.mask = p.mask;
  a.pm_cap = p.pm_cap;
  a.dev_status = p.dev_status;
  a.pm_col_blocks = 1;
  int64_t pm_blocks = 0;
  if (p.pos) {
    const int64_t width = static_cast<int64_t>(p.Lb) + p.k + 1;
    a.pm_col_blocks = static_cast<uint32_t>((width + 4 * kTpb - 1) / (4 * kTpb));
    pm_blocks = static_cast<int64_t>(a.pm_col_blocks) * p.B;
  }
  a.tok_col_blocks = p.batch_tok ? static_cast<uint32_t>((static_cast<int64_t>(p.Lb) + 1 + 4 * kTpb - 1) / (4 * kTpb)) : 1u;
  const int64_t tok_blocks = static_cast<int64_t>(a.tok_col_blocks) * p.B;
  const int64_t extra = pm_blocks + tok_blocks;
  const int64_t nspans = p.Lb > 0 ? static_cast<int64_t>(p.L) * 2 * p.B * p.H : 0;
  a.misaligned = !split_spans_aligned<kPieces, kSplit>(p.batch, a.batch_span_vecs);
  const int64_t chunks = split_blocks<kPieces, kTpb, kSplit>(static_cast<int64_t>(p.Lb) * a.vpc, a.misaligned != 0);
  a.chunks = static_cast<uint32_t>(chunks > 0 ? chunks : 1);
  const int64_t max_blocks = max_launch_items() / kTpb - extra;
  const int64_t per_launch = max_blocks / a.chunks;
  if (per_launch < 1) return hipErrorInvalidConfiguration;
  for (int64_t s0 = 0; s0 == 0 || s0 < nspans; s0 += per_launch) {
    const int64_t ns = nspans - s0 < per_launch ? nspans - s0 : per_launch;
    const bool first = s0 == 0;
    a.span_base = static_cast<uint32_t>(s0);
    a.pm_blocks = first ? static_cast<uint32_t>(pm_blocks) : 0u;
    a.tok_blocks = first ? static_cast<uint32_t>(tok_blocks) : 0u;
    const int64_t blocks = ns * a.chunks + (first ? extra : 0);
    if (blocks > 0) {
      hipLaunchKernelGGL(gather_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTpb), 0, stream, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if (ns <= 0) break;
  }
  return hipSuccess;
}

hipError_t launch_writeback(const WritebackLaunch& p, hipStream_t stream) {
  WritebackArgs a{};
  a.batch = static_cast<const u32x4*>(p.batch);
  a.pool = static_cast<u32x4*>(p.pool);
  a.vpc = p.D / 8;
  a.batch_span_vecs = p.batch_cap * a.vpc;
  a.pool_span_vecs = p.pool_cap * a.vpc;
  a.N = p.N;
  a.B = p.B;
  a.H = p.H;
  a.k = p.k;
  a.Lb = p.Lb;
  a.pool_cap = p.pool_cap;
  a.pads = p.pads;
  a.tokens = p.tokens;
  a.n_acc = p.n_acc;
  a.slots = p.slots;
  a.pool_tok = p.pool_tok;
  a.pool_tok_stride = p.pool_tok_stride;
  a.lens = p.lens;
  a.batch_tok = p.batch_tok;
  a.btok_stride = p.btok_stride;
  a.dev_status = p.dev_status;
  const int64_t nspans = static_cast<int64_t>(p.L) * 2 * p.B * p.H;
  const int64_t extra = p.B;
  int64_t chunks = 1;
  a.misaligned = !p.append_only && !split_spans_aligned<kPieces, kSplit>(p.pool, a.pool_span_vecs);
  if (!p.append_only)
    chunks = split_blocks<kPieces, kTpb, kSplit>((static_cast<int64_t>(p.Lb) + p.k + 1) * a.vpc, a.misaligned != 0);
  a.chunks = static_cast<uint32_t>(chunks);
  const int64_t max_blocks = max_launch_items() / kTpb - extra;
  const int64_t per_launch = max_blocks / chunks;
  if (per_launch < 1) return hipErrorInvalidConfiguration;
  for (int64_t s0 = 0; s0 == 0 || s0 < nspans; s0 += per_launch) {
    const int64_t ns = nspans - s0 < per_launch ? nspans - s0 : per_launch;
    const bool first = s0 == 0;
    a.span_base = static_cast<uint32_t>(s0);
    a.meta_blocks = first ? static_cast<uint32_t>(extra) : 0u;
    const int64_t blocks = ns * chunks + (first ? extra : 0);
    if (blocks > 0) {
      if (p.append_only)
        hipLaunchKernelGGL(writeback_append_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTpb), 0, stream, a);
      else
        hipLaunchKernelGGL(writeback_full_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTpb), 0, stream, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if (ns <= 0) break;
  }
  return hipSuccess;
}

}  // namespace specdec
