// Internal launch interface between the C-ABI layer (specdec_api.cpp) and the
// HIP kernels (specdec_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specdec {

constexpr int kThreads = 256;          // every kernel: 4 wavefronts of 64
constexpr size_t kWsHeaderBytes = 256; // reserved, keeps the partial maxima 256-byte aligned
constexpr int64_t kMaxVerifyChunks = 64;  // workgroups per logit row in the verify scan

struct VerifyLaunch {
  const void* logits;
  int dtype;                 // 0 f32, 1 bf16, 2 f16
  const int32_t* draft;
  const int32_t* pad_in;
  int32_t B, k, V, W_in;
  int32_t* tokens;
  int32_t* n_acc;
  int32_t* bonus;            // may be null
  int32_t* pad_out;
  int32_t* w_new;
  void* workspace;           // [header][partial maxima: B*(k+1)*chunks uint64][order table]
  uint32_t* dev_status;      // may be null
  bool write_order = false;  // also write the in-place realignment order into the workspace
};

// In-place realignment order, written by the verification merge into the
// workspace after the partial maxima: one int4 per row (row, pad_in,
// pad_out, new length), the moving rows first in classes of decreasing
// length (the cache's order within a class), then the rows that do not move
// or whose pad_in is out of range (written with pad_out = pad_in: nothing
// to do).
constexpr int kMaxOrderClasses = 8;
// Byte offset of the order table in a verification workspace, and its size.
int64_t order_offset(int64_t B, int64_t k, int64_t V);
int64_t order_bytes(int64_t B);
int64_t order_bytes(int64_t B);

struct RealignLaunch {
  const void* src;
  void* dst;
  int64_t src_cap, dst_cap;
  int32_t L, B, H, D;
  int32_t k, W_in;
  const int32_t* pad_in;
  const int32_t* n_acc;
  const int32_t* w_new;
  uint32_t* dev_status;
  bool in_place;
  // fused position ids / mask (pos == nullptr: none)
  int64_t* pos;
  uint8_t* mask;
  int64_t pm_cap;
  const int32_t* pad_out;    // verify's pad_out; used only by the fused pos/mask blocks
  // token row S (s_in == nullptr: none); s_out == s_in: in place
  const int32_t* s_in;
  int32_t* s_out;
  int64_t s_in_stride, s_out_stride;
  const int32_t* tokens;
  int32_t pad_id;
  // in place: the order table written by verification (NULL: the cache's order)
  const int32_t* order = nullptr;
  // words the launch zeroes in one extra workgroup (NULL: none)
  uint32_t* clear_words = nullptr;
  uint32_t clear_count = 0;
};

struct PosmaskLaunch {
  const int32_t* pad_out;
  const int32_t* w_new;
  int32_t B, k;
  int64_t* pos;
  uint8_t* mask;
  int64_t pm_cap;
  int64_t col_bound;         // upper bound of w_new + k + 1 known on the host
  uint32_t* dev_status;
};

// Verify chunking chosen on the host: elements of one logit row per
// workgroup, and workgroups per row.
int64_t verify_chunk_elems(int64_t rows, int64_t V);
int64_t verify_chunks(int64_t rows, int64_t V);


// EXSpec batch gather (pool slots -> left-padded batch, token rows, paddings,
// position ids / mask).
struct GatherLaunch {
  const void* pool;
  int64_t pool_cap;
  int32_t N;
  const int32_t* pool_tok;     // may be null when batch_tok is
  int64_t pool_tok_stride;
  const int32_t* lens;
  const int32_t* slots;
  int32_t L, B, H, D;
  int32_t Lb, k;
  void* batch;
  int64_t batch_cap;
  int32_t* batch_tok;          // may be null
  int64_t btok_stride;
  int32_t pad_id;
  int32_t* pads;
  int64_t* pos;                // may be null (then mask is too)
  uint8_t* mask;
  int64_t pm_cap;
  uint32_t* dev_status;
};

// EXSpec write-back (batch rows -> pool slots).
struct WritebackLaunch {
  const void* batch;
  int64_t batch_cap;
  const int32_t* pads;
  const int32_t* tokens;
  const int32_t* n_acc;
  const int32_t* slots;
  int32_t L, B, H, D;
  int32_t k, Lb;
  void* pool;
  int64_t pool_cap;
  int32_t N;
  int32_t* pool_tok;
  int64_t pool_tok_stride;
  int32_t* lens;
  int32_t* batch_tok;          // may be null
  int64_t btok_stride;
  bool append_only;
  uint32_t* dev_status;
};

// Stochastic verification (speculative sampling at temperature T > 0).
struct SampleLaunch {
  const void* logits;        // [B][k+1][V]
  const void* draft_logits;  // [B][k][V]
  int dtype;
  const int32_t* draft;
  const int32_t* pad_in;
  const float* u_accept;
  const float* u_sample;
  float c;                   // log2(e) / T
  int32_t B, k, V, W_in;
  int32_t* tokens;
  int32_t* n_acc;
  int32_t* bonus;
  int32_t* pad_out;
  int32_t* w_new;
  void* workspace;           // [header][chunk (max, sum): B*(2k+1)*chunks float2][masses, last indices]
  uint32_t* dev_status;
};

// Chunking of the stochastic verification's row statistics.
int64_t sample_chunk_elems(int64_t rows, int64_t V);
int64_t sample_chunks(int64_t rows, int64_t V);
int64_t sample_mass_chunk_elems(int64_t B, int64_t V);
hipError_t launch_verify_sample(const SampleLaunch& p, hipStream_t stream);
// The launches of launch_verify_sample: the row statistics over every target
// and draft logit, then the accept tests, masses and draws.
hipError_t launch_sample_stats(const SampleLaunch& p, hipStream_t stream);
hipError_t launch_sample_finish(const SampleLaunch& p, hipStream_t stream);

// Family A rollback (truncation to the batch-minimum accepted count).
struct RollbackLaunch {
  const int32_t* tokens;
  const int32_t* n_acc_in;
  const int32_t* pad_in;
  int32_t B, k, W_in;
  int32_t* n_acc_out;
  int32_t* bonus_out;
  int32_t* pad_out;
  int32_t* w_new;
  uint32_t* dev_status;
};

// Family B rollback (compaction of a flat [L][2][T][H][D] cache).
struct VarlenLaunch {
  const void* src;
  void* dst;
  int64_t src_T, dst_T;
  int32_t L, H, D;
  const int32_t* cu_in;
  const int32_t* n_acc;
  int32_t B, k, max_len;
  int32_t* cu_out;
  int64_t* pos;              // may be null
  uint32_t* dev_status;
};

hipError_t launch_rollback(const RollbackLaunch& p, hipStream_t stream);
hipError_t launch_varlen_rollback(const VarlenLaunch& p, hipStream_t stream);

hipError_t launch_gather(const GatherLaunch& p, hipStream_t stream);
hipError_t launch_writeback(const WritebackLaunch& p, hipStream_t stream);

// Message of the calling thread's last failure (specdec_last_error), for
// entry points defined outside the main API source.
void set_last_error(const char* msg);
void clear_last_error();

// Largest number of work-items one dispatch may hold (2^32 - 1, or lower when
// the environment variable SPECDEC_MAX_LAUNCH_ITEMS asks for it, to exercise
// the split of a grid over several launches).
int64_t max_launch_items();

hipError_t launch_verify(const VerifyLaunch& p, hipStream_t stream);
// The two launches of launch_verify: the vocabulary scan (partial maxima),
// then the one-workgroup merge (tokens, accepted counts, width, paddings).
hipError_t launch_verify_scan(const VerifyLaunch& p, hipStream_t stream);
hipError_t launch_verify_finalize(const VerifyLaunch& p, hipStream_t stream);
// Greedy verification in one launch (one workgroup per logit row): for
// batches of at most kMaxFusedVerifyRows rows of at most
// kMaxFusedVerifyRowBytes bytes each (verify_fused_fits).  `counts` holds
// 1 + 2 * kMaxFusedVerifyRows words: the batch completion count, the B
// per-sequence counts, then (from word 1 + kMaxFusedVerifyRows) the new
// lengths.  The first B + 1 words must be zero on entry and are left
// non-zero.
constexpr int64_t kMaxFusedVerifyRows = 4096;
constexpr int64_t kMaxFusedVerifyRowBytes = 16 * 1024;
bool verify_fused_fits(int64_t B, int64_t k, int64_t V, int dtype);
hipError_t launch_verify_fused(const VerifyLaunch& p, uint32_t* counts, hipStream_t stream);
hipError_t launch_realign(const RealignLaunch& p, hipStream_t stream);
hipError_t launch_posmask(const PosmaskLaunch& p, hipStream_t stream);
// Token row only (RealignLaunch's cache fields are ignored).
hipError_t launch_tokens(const RealignLaunch& p, hipStream_t stream);
hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream);

}  // namespace specdec
