/*
 * specdec.h — C ABI of libspecdec.so: one step of greedy batch speculative
 * decoding under the EqSpec method (arXiv 2510.22876) on AMD MI355X (gfx950).
 *
 * One step = greedy batch verification (Algorithm 3, BatchVerify) followed by
 * unpad-append-repad realignment of a left-padded contiguous KV cache
 * (Section 3.1, Eq. (1) and Eq. (2); Theorem B.1) and the rebuild of position
 * ids and the attention mask (invariant I2), so that rectangular alignment
 * (I1) and position / KV-cache correspondence (I2) hold after the step.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer argument that names a tensor is a DEVICE pointer (memory
 *   from hipMalloc or a torch CUDA/HIP tensor) unless it says "host".  The
 *   caller owns every buffer; the library never allocates, frees or keeps a
 *   pointer after the call returns.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *   work is enqueued on it and the call returns without waiting, except where
 *   a host output is requested.
 * - Return value: a specdec_status_t.  Problems the host can see (NULL
 *   pointers, sizes out of range, misalignment, overlapping buffers, a short
 *   workspace) are reported before anything is enqueued; nothing is written
 *   then.  SPECDEC_ERR_HIP reports a failed HIP call.  specdec_last_error()
 *   gives the message of the last failure on the calling thread.
 * - Device-resident values (pad_in, n_acc, w_new, pad_out) cannot be checked
 *   by the host.  Kernels check them before any memory access they steer; a
 *   row whose values are out of range is left untouched and a bit is set in
 *   the optional `dev_status` word (device uint32, may be NULL; bits are
 *   OR-ed in and never cleared by the library).
 * - No output (a destination cache or token row and the `dev_status` word
 *   included) may overlap an input or another output; inputs may overlap
 *   each other.  A cache or token row realigned in place is one buffer, read
 *   and written by the same call.  An overlap is SPECDEC_ERR_INVALID_ARGUMENT.
 * - One launch holds fewer than 2^32 work-items; larger caches are moved by
 *   several launches of the same kernel on the same stream.  The environment
 *   variable SPECDEC_MAX_LAUNCH_ITEMS (a positive integer) lowers that cap, so
 *   the multi-launch path can be tested at small sizes; results are the same.
 *
 * Terms: B rows, k draft tokens per row, V vocabulary entries.  W_in is the
 * width of the cache handed to the step, counted in cache columns and
 * including the k+1 columns of the verify window; L = W_in - (k+1) is the
 * width of the cache before the window.  Row i holds c_i = L - pad_in[i]
 * cached entries in columns [pad_in[i], L) and the entries of the verify
 * window [pending token, d_1 .. d_k] in columns [L, W_in).  Logit row r of
 * sequence i scores the token that follows window slot r.
 */
#ifndef SPECDEC_H
#define SPECDEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPECDEC_ABI_VERSION 5

typedef enum {
  SPECDEC_OK = 0,
  SPECDEC_ERR_INVALID_ARGUMENT = 1, /* NULL pointer, size out of range, overlap   */
  SPECDEC_ERR_UNSUPPORTED = 2,      /* dtype, alignment or head size not handled */
  SPECDEC_ERR_HIP = 3,              /* a HIP runtime call failed                 */
  SPECDEC_ERR_WORKSPACE = 4         /* workspace missing or too small            */
} specdec_status_t;

typedef enum { SPECDEC_F32 = 0, SPECDEC_BF16 = 1, SPECDEC_F16 = 2 } specdec_dtype_t;

/* Bits OR-ed into *dev_status by the kernels. */
#define SPECDEC_DEV_BAD_PAD_IN 0x1u  /* pad_in[i] outside [0, L]                        */
#define SPECDEC_DEV_BAD_ACCEPT 0x2u  /* n_acc[i] outside [0, k]                         */
#define SPECDEC_DEV_BAD_WIDTH 0x4u   /* w_new outside [1, W_in] or shorter than a row   */
#define SPECDEC_DEV_BAD_PAD_OUT 0x8u /* pad_out[i] outside [0, w_new] or pos/mask short */
#define SPECDEC_DEV_BAD_SLOT 0x10u   /* pool slot outside [0, N), or its length does not
                                        fit the batch width, the pool or its token row */
#define SPECDEC_DEV_SLOT_LEN 0x20u   /* write-back: lens[slot] != Lb - pads[i] on entry */
#define SPECDEC_DEV_BAD_UNIFORM 0x40u /* a uniform outside [0, 1) (clamped into it)       */

/* Limits checked by the host. */
#define SPECDEC_MAX_B 65536
#define SPECDEC_MAX_K 64
#define SPECDEC_MAX_ROWS 1048576      /* B*(k+1)                                   */
#define SPECDEC_MAX_WIDTH 16777216    /* W_in, cap and pm_cap                      */
#define SPECDEC_MAX_D 4096
#define SPECDEC_MAX_SAMPLE_V 8388608  /* vocabulary of stochastic verification          */
#define SPECDEC_NOALLOC_SCRATCH_BYTES 4194304  /* library scratch of specdec_step_noalloc */

/* A bf16 KV cache [L][2][B][H][cap][D], contiguous, D fastest.  One
 * (layer, K/V, row, head) "span" is cap*D contiguous elements.  `data` is a
 * device pointer, 16-byte aligned; D must be a multiple of 8 (rows of 16-byte
 * vectors). */
typedef struct specdec_kv {
  void* data;
  int32_t L, B, H, D;
  int64_t cap;
} specdec_kv_t;

/* ABI version of the loaded library (SPECDEC_ABI_VERSION at build time). */
int32_t specdec_abi_version(void);

/* Message of the last failure on the calling thread ("" if none).  The
 * string stays valid until the next call on this thread. */
const char* specdec_last_error(void);

/* Bytes of device workspace specdec_verify_greedy / specdec_step need for a
 * batch of B rows, k drafts and a vocabulary of V (0 on invalid sizes).  The
 * workspace holds per-workgroup partial maxima of the argmax and, for an
 * in-place specdec_step, the order in which the realignment takes the rows
 * (longest moving rows first); it needs no initialisation and its contents
 * after a call are unspecified.  The size does not depend on the logit
 * dtype, so no dtype argument is taken.  One
 * workspace serves one in-flight call: calls that share a workspace must be
 * ordered (same stream). */
size_t specdec_workspace_bytes(int32_t B, int32_t k, int32_t V);

/* Zero a workspace on `stream` with a kernel (never needed for correctness;
 * provided for callers that want deterministic scratch contents). */
specdec_status_t specdec_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/*
 * Greedy batch verification (Algorithm 3) and the new width and paddings
 * (Eq. (1), Eq. (2)).
 *
 *   logits    [B][k+1][V] of `dtype` (SPECDEC_F32 / _BF16 / _F16), contiguous,
 *             aligned to its element size.
 *   draft     int32 [B][k]: the draft tokens d_1..d_k of each row.
 *   pad_in    int32 [B]: left padding of each row, 0 <= pad_in[i] <= L.
 *   tokens    int32 [B][k+1] out: tokens[i][r] = lowest index of the maximum of
 *             logits[i][r][:] (-0.0 == +0.0; a NaN ranks above every number,
 *             the first NaN wins).
 *   n_acc     int32 [B] out: number of accepted drafts, the first r < k with
 *             draft[i][r] != tokens[i][r], else k.
 *   bonus     int32 [B] out (may be NULL): tokens[i][n_acc[i]], the target's
 *             correction / bonus token (never a draft token).
 *   pad_out   int32 [B] out: new left padding w_new - (c_i + n_acc[i] + 1);
 *             -1 for a row whose pad_in is out of range.
 *   w_new     int32 [1] out: new shared width L' = max_i (c_i + n_acc[i] + 1)
 *             over rows with a valid pad_in (0 if none).  L' <= W_in.
 *   workspace device memory of specdec_workspace_bytes(B, k, V) bytes,
 *             8-byte aligned.
 * B = 0 is a no-op.  Limits: 1 <= V < 2^31, 0 <= k <= SPECDEC_MAX_K,
 * B <= SPECDEC_MAX_B, B*(k+1) <= SPECDEC_MAX_ROWS, k+1 <= W_in <= SPECDEC_MAX_WIDTH.
 * The outputs and the workspace must not overlap each other or the inputs
 * (a decode loop keeps pad_in and pad_out in separate buffers and swaps
 * them); an overlap is SPECDEC_ERR_INVALID_ARGUMENT.
 */
specdec_status_t specdec_verify_greedy(const void* logits, int32_t dtype, const int32_t* draft,
                                       const int32_t* pad_in, int32_t B, int32_t k, int32_t V,
                                       int32_t W_in, int32_t* tokens, int32_t* n_acc,
                                       int32_t* bonus, int32_t* pad_out, int32_t* w_new,
                                       void* workspace, size_t workspace_bytes,
                                       uint32_t* dev_status, void* stream);

/*
 * Stochastic verification at temperature T > 0: the counterpart of
 * specdec_verify_greedy for sampled decoding.  At T > 0, output equivalence
 * means the emitted tokens follow the target model's distribution (the
 * equivalence requirement of Section 2), which speculative sampling keeps
 * (Chen et al. 2023; Leviathan et al. 2023).  With p_r = softmax(logits[i][r]
 * / T) and q_r = softmax(draft_logits[i][r] / T):
 *   draft r is accepted iff u_accept[i][r] * q_r(draft[i][r]) <
 *   p_r(draft[i][r]); n_acc[i] is the first rejected slot (k if none);
 *   at a rejection the correction token is drawn from max(0, p_r - q_r)
 *   (normalised; p_r if that has no mass), after k acceptances the bonus
 *   from p_k, by inversion with u_sample[i]: the smallest index whose
 *   cumulative weight exceeds u_sample[i] times the total.
 * tokens[i][0 .. n_acc[i]] are the accepted drafts and the drawn token (later
 * entries -1), bonus[i] the drawn token; pad_out and w_new as in greedy
 * verification (Eq. (1), Eq. (2)), so the realignment entry points apply
 * unchanged.
 *
 *   logits        [B][k+1][V], draft_logits [B][k][V], both of `dtype`
 *                 (SPECDEC_F32 / _BF16 / _F16), contiguous, aligned to the
 *                 element size.  Every row needs a finite maximum; -inf
 *                 entries have probability 0; NaN or +inf give unspecified
 *                 tokens (never an out-of-bounds access).
 *   u_accept      float [B][k], u_sample float [B]: uniforms in [0, 1) drawn by
 *                 the caller (values outside are clamped into [0, 1) and
 *                 flagged SPECDEC_DEV_BAD_UNIFORM).
 *   temperature   T > 0, finite, with log2(e) / T finite in fp32.
 *   workspace     specdec_sample_workspace_bytes(B, k, V) bytes, 8-byte
 *                 aligned; no initialisation needed.
 * Arithmetic is fp32 (exp2 of scaled differences from the row maximum, sums
 * in a fixed parallel order): a decision whose fp64 margin is within the
 * fp32 rounding of these sums may differ from an fp64 evaluation.
 * Limits as specdec_verify_greedy, with B*(2k+1) <= SPECDEC_MAX_ROWS and
 * V <= SPECDEC_MAX_SAMPLE_V; outputs and workspace must not overlap each
 * other or the inputs, as there.
 */
size_t specdec_sample_workspace_bytes(int32_t B, int32_t k, int32_t V);

specdec_status_t specdec_verify_sample(const void* logits, const void* draft_logits, int32_t dtype,
                                       const int32_t* draft, const int32_t* pad_in,
                                       const float* u_accept, const float* u_sample,
                                       float temperature, int32_t B, int32_t k, int32_t V,
                                       int32_t W_in, int32_t* tokens, int32_t* n_acc,
                                       int32_t* bonus, int32_t* pad_out, int32_t* w_new,
                                       void* workspace, size_t workspace_bytes,
                                       uint32_t* dev_status, void* stream);

/*
 * Unpad-append-repad of the KV cache (Section 3.1; Theorem B.1's relocation).
 *
 * For every (layer, K/V, row i, head) span, with c_i = L - pad_in[i],
 * a_i = n_acc[i] + 1 and p'_i = w_new - (c_i + a_i): destination columns
 * [0, p'_i) become +0.0 and destination column j in [p'_i, w_new) receives
 * source column j - (p'_i - pad_in[i]), bit for bit.  Source columns kept are
 * [pad_in[i], L + a_i); window columns of rejected drafts are dropped.
 * Destination columns [w_new, cap) are left as they are.
 *
 *   src, dst  KV descriptors with equal L, B, H, D; src->cap >= W_in,
 *             dst->cap >= W_in (w_new <= W_in always holds).
 *             dst->data == src->data (same cap): in place.  In place requires
 *             the input's pad columns [0, pad_in[i]) to be +0.0 (they are
 *             not rewritten); it moves only rows whose padding changes.
 *             Otherwise the two caches must not overlap.
 *   pad_in, n_acc  int32 [B] (device); w_new int32 [1] (device): the outputs
 *             of specdec_verify_greedy for this step; none of them may lie
 *             inside dst.
 */
specdec_status_t specdec_realign_kv(const specdec_kv_t* src, const specdec_kv_t* dst, int32_t k,
                                    int32_t W_in, const int32_t* pad_in, const int32_t* n_acc,
                                    const int32_t* w_new, uint32_t* dev_status, void* stream);

/*
 * Position ids and attention mask of invariant I2 for the realigned batch.
 *
 * For columns j in [0, w_new + k + 1) (the realigned cache plus the next
 * verify window): mask[i][j] = (j >= pad_out[i]), pos[i][j] =
 * max(0, #content columns q <= j - 1) = max(0, j - pad_out[i]).  Columns
 * [w_new + k + 1, pm_cap) are left as they are.
 *
 *   pad_out   int32 [B], w_new int32 [1] (device).
 *   pos       int64 [B][pm_cap] out, 8-byte aligned; mask uint8 [B][pm_cap] out.
 *   pm_cap    row stride of pos and mask; must be >= w_new + k + 1 (checked on
 *             the device; rows that do not fit are skipped and flagged).
 * pos and mask must not overlap each other, pad_out or w_new (nor, in
 * specdec_step, any other buffer of the step).
 */
specdec_status_t specdec_build_posmask(const int32_t* pad_out, const int32_t* w_new, int32_t B,
                                       int32_t k, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                       uint32_t* dev_status, void* stream);

/*
 * Realignment of the token row S with the same offsets (Alg. 1, phase 3:
 * S[i] <- S[i] + A[i] + B[i], then fresh left padding).
 *
 * Row i of S before the step holds pad_in[i] pad tokens and then c_i + 1
 * tokens (the c_i cached tokens and the pending token), L + 1 columns in all.
 * After the step row i holds pad_out[i] = w_new - (c_i + n_acc[i] + 1) copies
 * of pad_id, those c_i + 1 tokens, then tokens[i][0 .. n_acc[i]] (the accepted
 * drafts and the bonus token): w_new + 1 columns.  Columns beyond are left
 * as they are.
 *
 *   s_in      int32 [B][s_in_stride], s_in_stride >= W_in - k (device).
 *   s_out     int32 [B][s_out_stride], s_out_stride >= W_in + 1 (device);
 *             s_out == s_in with equal strides: in place (the input's columns
 *             [0, pad_in[i]) need not hold pad_id); otherwise the two must not
 *             overlap.
 *   tokens    int32 [B][k+1], pad_in, n_acc int32 [B], w_new int32 [1]: the
 *             outputs of specdec_verify_greedy for this step; none of them
 *             may lie inside s_out.
 */
specdec_status_t specdec_realign_tokens(const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                                        int64_t s_out_stride, const int32_t* tokens,
                                        const int32_t* pad_in, const int32_t* n_acc,
                                        const int32_t* w_new, int32_t B, int32_t k, int32_t W_in,
                                        int32_t pad_id, uint32_t* dev_status, void* stream);

/*
 * One EqSpec step after the forwards (Algorithm 1, phases 2 and 3: batch
 * verification, then unpad-append-repad of the cache, the token row and the
 * attention inputs so that I1 and I2 hold for the next forward), on one
 * stream: specdec_verify_greedy, then one fused launch of the cache
 * realignment, the position ids / mask and (when s_in is not NULL) the token
 * row realignment.  In place, the verification also writes into the
 * workspace the order in which the realignment takes the rows (the longest
 * moving rows first).  Arguments as above; pm_cap must be
 * >= W_in + k + 1.  Every output (tokens, n_acc, bonus, pad_out, w_new, the
 * workspace, pos, mask, dst, s_out, dev_status) stands apart from every
 * input (logits, draft, pad_in, src, s_in) and from the other outputs,
 * except that dst may be src and s_out may be s_in (in place).  If
 * `w_new_host` (host int32*) is not NULL, the stream is synchronised and L'
 * is copied there.
 */
specdec_status_t specdec_step(const void* logits, int32_t dtype, const int32_t* draft,
                              const int32_t* pad_in, int32_t B, int32_t k, int32_t V,
                              int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                              int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                              int32_t* w_new, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                              const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                              int64_t s_out_stride, int32_t pad_id,
                              void* workspace, size_t workspace_bytes, uint32_t* dev_status,
                              int32_t* w_new_host, void* stream);

/*
 * specdec_step without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, outputs and checks as
 * specdec_step, minus workspace / workspace_bytes.
 *
 * The step's scratch is a library-owned device array of
 * SPECDEC_NOALLOC_SCRATCH_BYTES, one copy per device, held until the process
 * ends; its address is looked up once per device (on the first call with
 * that device current) and nothing is allocated or freed, ever.  The
 * device's first step that passes every argument check also enqueues, ahead
 * of its own kernels, one kernel that clears the array's completion counts;
 * a call that fails a check enqueues nothing.
 *
 * Batches of at most 4096 logit rows (B*(k+1)) of at most 16 KB each
 * (V*4 bytes for f32, V*2 for bf16 / f16) verify in ONE launch: a workgroup
 * per row, and the last row of a sequence, then the last sequence, to finish
 * merges (counted in the scratch; the realignment launch clears the counts
 * again).  The step is then two launches.  Larger batches verify in the scan
 * and merge launches of specdec_step, with the partial maxima in the
 * scratch; one whose partial maxima need more than
 * SPECDEC_NOALLOC_SCRATCH_BYTES - 64 KiB (specdec_workspace_bytes(B, k, V))
 * is rejected with SPECDEC_ERR_WORKSPACE before anything is enqueued.  The
 * outputs are the same bits as specdec_step's either way.
 *
 * The stream must belong to the current device (SPECDEC_ERR_INVALID_ARGUMENT
 * otherwise).  Every call on one device shares that device's scratch, so
 * calls on one device that may overlap in time (on different streams, or
 * graph replays running concurrently) race and give unspecified results;
 * order them.  A later step that runs alone is correct again: each step's
 * realignment clears the counts it and any racing call left behind.
 */
specdec_status_t specdec_step_noalloc(const void* logits, int32_t dtype, const int32_t* draft,
                                      const int32_t* pad_in, int32_t B, int32_t k, int32_t V,
                                      int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                                      int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                                      int32_t* w_new, int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                      const int32_t* s_in, int64_t s_in_stride, int32_t* s_out,
                                      int64_t s_out_stride, int32_t pad_id, uint32_t* dev_status,
                                      int32_t* w_new_host, void* stream);

/* ---- EXSpec (Algorithm 2): sequence pool, batch gather and write-back ---------
 *
 * EXSpec keeps every sequence unpadded in its own slot of a pool and forms each
 * step's batch from a window of active sequences (Section 3.2, "Cross-Batch
 * Scheduling"; Appendix: EXSpec, Algorithm 2).  The pool cache has the KV
 * layout with one row per slot: [L][2][N][H][pool_cap][D] (pool->B = N);
 * slot s holds its lens[s] cached entries in columns [0, lens[s]).  The pool
 * token rows are int32 [N][pool_tok_stride]; slot s holds its lens[s] cached
 * tokens and then its pending token in columns [0, lens[s]].
 */

/*
 * GetBatch (Algorithm 2, phase 1): gather the rows `slots` of the pool into a
 * batch left-padded to width Lb.  Same-length rows concatenate with no padding
 * (the case the scheduler looks for); otherwise this is the unpad-repad
 * fallback.  For row i with slot s = slots[i] and n = lens[s]:
 *   pads[i] = Lb - n;
 *   batch columns [0, pads[i]) of every (layer, K/V, head) span become +0.0 and
 *   column j in [pads[i], Lb) receives pool column j - pads[i] of slot s;
 *   batch_tok[i][0, pads[i]) = pad_id, batch_tok[i][pads[i] + j] =
 *   pool_tok[s][j] for j in [0, n]  (Lb + 1 columns);
 *   pos / mask over columns [0, Lb + k + 1) as in specdec_build_posmask with
 *   pad_out = pads and w_new = Lb (the mask of the draft and verify forwards).
 * Batch columns [Lb, cap) and token columns beyond Lb are left as they are.
 *
 *   pool      the pool cache (pool->B = N slots); pool_tok int32 [N][pool_tok_stride].
 *   lens      int32 [N] (device): cached entries per slot.
 *   slots     int32 [B] (device): the batch's slots, row order.  Slots must be
 *             distinct (not checked: repeated slots are gathered twice).
 *   Lb        batch width (host), >= lens[slots[i]] for every row.
 *   batch     cache [L][2][B][H][cap][D] with equal L, H, D, cap >= Lb; must
 *             not overlap the pool.
 *   batch_tok int32 [B][btok_stride], btok_stride >= Lb + 1; may be NULL.
 *   pads      int32 [B] out; -1 for a row that was skipped.
 *   pos, mask int64 / uint8 [B][pm_cap], pm_cap >= Lb + k + 1; may be NULL
 *             (both, then k is not used).
 * A row whose slot is outside [0, N) or whose length is outside [0, Lb], above
 * pool_cap or above pool_tok_stride - 1 is skipped (no byte of it written) and
 * flagged SPECDEC_DEV_BAD_SLOT.  The outputs (batch cache, batch_tok, pads,
 * pos, mask) must not overlap each other or the inputs (pool cache, pool_tok,
 * lens, slots): SPECDEC_ERR_INVALID_ARGUMENT.
 */
specdec_status_t specdec_gather_batch(const specdec_kv_t* pool, const int32_t* pool_tok,
                                      int64_t pool_tok_stride, const int32_t* lens,
                                      const int32_t* slots, int32_t B, int32_t Lb, int32_t k,
                                      const specdec_kv_t* batch, int32_t* batch_tok,
                                      int64_t btok_stride, int32_t pad_id, int32_t* pads,
                                      int64_t* pos, uint8_t* mask, int64_t pm_cap,
                                      uint32_t* dev_status, void* stream);

#define SPECDEC_WRITEBACK_FULL 0   /* copy the row's whole unpadded cache            */
#define SPECDEC_WRITEBACK_APPEND 1 /* copy only the row's n_acc[i] + 1 new entries     */

/*
 * Write-back (Algorithm 2, phase 4) after verification of a gathered batch
 * (rows end at column Lb, row i has pads[i] columns of padding, the verify
 * window is in columns [Lb, Lb + k + 1)).  For row i with slot s = slots[i],
 * n = Lb - pads[i] and a = n_acc[i] + 1:
 *   Pool[s] <- Pool[s] + A[i] + B[i]: pool_tok[s][n + 1 + r] = tokens[i][r]
 *     for r in [0, a) (the accepted drafts and the bonus token);
 *   Pool.KV[s] <- KV[i]: pool columns [0, n + a) of slot s receive batch
 *     columns [pads[i], Lb + a) of row i (SPECDEC_WRITEBACK_FULL), or only
 *     columns [n, n + a) receive batch columns [Lb, Lb + a)
 *     (SPECDEC_WRITEBACK_APPEND: the same result whenever the slot still holds
 *     the n entries the row was gathered from, which Algorithm 2 guarantees:
 *     the forwards only append to the batch);
 *   lens[s] = n + a;
 *   when batch_tok is not NULL: batch_tok[i][Lb + 1 + r] = tokens[i][r] for
 *     r in [0, a), so a batch kept for the next step (lazy realignment, all
 *     rows accepting alike) has its token rows extended as a new gather would.
 *
 *   batch     cache [L][2][B][H][cap][D], cap >= Lb + k + 1; must not overlap
 *             the pool.  pads int32 [B], tokens int32 [B][k+1], n_acc int32 [B]:
 *             from specdec_gather_batch and specdec_verify_greedy.
 *   slots     int32 [B], distinct (not checked: repeated slots leave those
 *             slots' contents unspecified; every access stays in bounds).
 *   pool, pool_tok, lens  as for specdec_gather_batch; written.
 *   batch_tok int32 [B][btok_stride], btok_stride >= Lb + k + 2; may be NULL.
 *   mode      SPECDEC_WRITEBACK_FULL or SPECDEC_WRITEBACK_APPEND.
 * A row with a slot outside [0, N), n_acc outside [0, k], pads outside
 * [0, Lb], or n + a above pool_cap or above pool_tok_stride - 1 is skipped and
 * flagged (SPECDEC_DEV_BAD_SLOT / _BAD_ACCEPT / _BAD_PAD_IN).  lens[s] !=
 * Lb - pads[i] on entry is flagged SPECDEC_DEV_SLOT_LEN (the row is still
 * written back).  The updated buffers (pool cache, pool_tok, lens, batch_tok)
 * must not overlap each other or the inputs (batch cache, pads, tokens, n_acc,
 * slots): SPECDEC_ERR_INVALID_ARGUMENT.
 */
specdec_status_t specdec_scatter_accepted(const specdec_kv_t* batch, const int32_t* pads,
                                          const int32_t* tokens, const int32_t* n_acc,
                                          const int32_t* slots, int32_t B, int32_t k, int32_t Lb,
                                          const specdec_kv_t* pool, int32_t* pool_tok,
                                          int64_t pool_tok_stride, int32_t* lens,
                                          int32_t* batch_tok, int64_t btok_stride, int32_t mode,
                                          uint32_t* dev_status, void* stream);

/*
 * The SequencePool scheduler of Algorithm 2 (host only; no GPU call).
 *
 * Holds N sequences with their lengths (cached entries), generated counts and
 * active flags.  The window is the first `window` active sequences in pool
 * order (sorted by initial length, ties by index, when sort_by_length; else
 * input order).  specdec_sched_next_batch picks, in this order:
 *   1. lazy realignment: the previous batch unchanged when its last step
 *      accepted the same number of drafts in every row (every offset of
 *      Eq. (2) is zero, Corollary B.4) and all its rows are still active;
 *   2. same-length grouping: window members bucketed by length; the bucket of
 *      the oldest window member if it has >= b members (b = min(batch, window
 *      members)), else the largest bucket with >= b members (ties: the
 *      shorter length); its first b members in pool order;
 *   3. fallback (unpad-repad): the first b window members.
 * The batch width is the longest row's length.  specdec_sched_commit records a
 * step's outcome: every row grows by n_acc[i] + 1; a sequence is deactivated
 * once it has generated >= max_new tokens or appended eos_id (eos_id >= 0).
 */
typedef struct specdec_sched specdec_sched_t; /* opaque */

typedef struct specdec_batch_info {
  int32_t B;           /* rows (0: no active sequence is left)               */
  int32_t width;       /* Lb: the longest row's length                       */
  int32_t same_length; /* 1: every row has the same length (no padding)      */
  int32_t reuse;       /* 1: the previous batch, unchanged (no gather needed) */
} specdec_batch_info_t;

/* lens: host int32 [N] initial cached entries per sequence (>= 0).  window,
 * batch >= 1, max_new >= 1.  *out receives the scheduler (free it with
 * specdec_sched_destroy). */
specdec_status_t specdec_sched_create(const int32_t* lens, int32_t N, int32_t window, int32_t batch,
                                      int32_t max_new, int32_t sort_by_length, int32_t eos_id,
                                      specdec_sched_t** out);
void specdec_sched_destroy(specdec_sched_t* s);

/* slots, lens: host int32 [batch] out (lens may be NULL): the batch's slots in
 * row order and their lengths.  Calling it again before a commit returns the
 * same batch. */
specdec_status_t specdec_sched_next_batch(specdec_sched_t* s, int32_t* slots, int32_t* lens,
                                          specdec_batch_info_t* info);

/* Outcome of the step run on the last batch: n_acc host int32 [B]; tokens host
 * int32 [B][k+1] (the predictions; row i appended tokens[i][0 .. n_acc[i]]),
 * may be NULL when eos_id < 0. */
specdec_status_t specdec_sched_commit(specdec_sched_t* s, const int32_t* n_acc,
                                      const int32_t* tokens, int32_t k);

/* Current lengths (host int32 [N] out), and the number of active sequences. */
specdec_status_t specdec_sched_lengths(const specdec_sched_t* s, int32_t* lens);
int32_t specdec_sched_active(const specdec_sched_t* s);

/*
 * The whole step with stochastic verification: specdec_verify_sample, then
 * the same fused realignment launch as specdec_step (cache, position ids /
 * mask, token row when s_in is not NULL).  Arguments as specdec_verify_sample
 * and specdec_step; the workspace is specdec_sample_workspace_bytes(B, k, V).
 */
specdec_status_t specdec_step_sample(const void* logits, const void* draft_logits, int32_t dtype,
                                     const int32_t* draft, const int32_t* pad_in,
                                     const float* u_accept, const float* u_sample,
                                     float temperature, int32_t B, int32_t k, int32_t V,
                                     int32_t W_in, const specdec_kv_t* src, const specdec_kv_t* dst,
                                     int32_t* tokens, int32_t* n_acc, int32_t* bonus,
                                     int32_t* pad_out, int32_t* w_new, int64_t* pos, uint8_t* mask,
                                     int64_t pm_cap, const int32_t* s_in, int64_t s_in_stride,
                                     int32_t* s_out, int64_t s_out_stride, int32_t pad_id,
                                     void* workspace, size_t workspace_bytes, uint32_t* dev_status,
                                     int32_t* w_new_host, void* stream);

/* ---- rollback: the other correct strategies of Section 2 -------------------- */

/*
 * Family A rollback (Section 2, "Family A: contiguous layout"): every row is
 * truncated to the batch-minimum accepted count m = min_i n_acc_in[i], so
 * every row appends tokens[i][0 .. m] and m + 1 cache entries; the width and
 * paddings follow Eq. (1) and Eq. (2) with a_i = m + 1 for every row, so all
 * offsets are equal (zero when the minimum input padding is 0, Corollary
 * B.4) and specdec_realign_kv in place moves no cached entry.  Correct, but
 * the verified tokens beyond m are discarded.
 *
 *   tokens      int32 [B][k+1], n_acc_in and pad_in int32 [B]: the outputs and
 *               inputs of specdec_verify_greedy / specdec_verify_sample.
 *   n_acc_out   int32 [B] out (all m; may equal n_acc_in), bonus_out int32 [B]
 *               out (tokens[i][m]), pad_out int32 [B] out (may equal pad_in),
 *               w_new int32 [1] out.
 * Rows with pad_in outside [0, W_in - k - 1] or n_acc_in outside [0, k] are
 * flagged (SPECDEC_DEV_BAD_PAD_IN / _BAD_ACCEPT), left out of m and the width,
 * and get pad_out = -1.
 */
specdec_status_t specdec_rollback(const int32_t* tokens, const int32_t* n_acc_in,
                                  const int32_t* pad_in, int32_t B, int32_t k, int32_t W_in,
                                  int32_t* n_acc_out, int32_t* bonus_out, int32_t* pad_out,
                                  int32_t* w_new, uint32_t* dev_status, void* stream);

/* A flat variable-length bf16 cache [L][2][T_cap][H][D], contiguous: the
 * rows of all sequences of a (layer, K/V) one after another, one row =
 * H*D elements (a multiple of 8).  `data` is a device pointer, 16-byte
 * aligned. */
typedef struct specdec_varlen {
  void* data;
  int32_t L, H, D;
  int64_t T_cap;
} specdec_varlen_t;

/*
 * Family B rollback (Section 2, "Family B: variable-length layout"): I1 does
 * not arise, but I2 requires the rejected entries to be rolled back.  Sequence
 * i holds rows [cu_in[i], cu_in[i+1]) of the flat buffer: its cached entries
 * followed by its k+1 verify window entries.  It keeps its first
 * cu_in[i+1] - cu_in[i] - (k - n_acc[i]) rows (the entries of the pending
 * token and the accepted drafts), compacted into dst at cu_out[i] =
 * the running sum of the kept lengths; pos[r] = the index of row r within its
 * sequence for r < cu_out[B].  Rows and positions beyond cu_out[B] are left
 * as they are.
 *
 *   src, dst    equal L, H, D; dst->T_cap >= src->T_cap; must not overlap.
 *   cu_in       int32 [B+1], nondecreasing, cu_in[B] <= src->T_cap.
 *   n_acc       int32 [B], from verification.
 *   max_len     host bound on every sequence's length cu_in[i+1] - cu_in[i]
 *               (sizes the grid), >= k + 1; values above src->T_cap act as
 *               src->T_cap.
 *   cu_out      int32 [B+1] out; pos int64 [pos_cap] out (may be NULL),
 *               pos_cap >= src->T_cap.
 * A sequence shorter than k + 1 rows or longer than max_len, outside the
 * buffer, or with n_acc outside [0, k] keeps no row and is flagged
 * (SPECDEC_DEV_BAD_WIDTH / _BAD_ACCEPT).  cu_out, pos and dst must not overlap
 * each other or cu_in, n_acc and src: SPECDEC_ERR_INVALID_ARGUMENT.
 */
specdec_status_t specdec_varlen_rollback(const specdec_varlen_t* src, const specdec_varlen_t* dst,
                                         const int32_t* cu_in, const int32_t* n_acc, int32_t B,
                                         int32_t k, int32_t max_len, int32_t* cu_out, int64_t* pos,
                                         int64_t pos_cap, uint32_t* dev_status, void* stream);

/*
 * Kernel timers (for measurement; off by default).  specdec_timing_enable
 * takes a mask of kernels (bit 1 << SPECDEC_KERNEL_*; 0 turns the timers
 * off).  For each selected kernel the library records a pair of HIP events on
 * the launch stream around its launch (verify: around its two launches).
 * specdec_timing_query waits for the recorded events, adds their durations to
 * the totals of `kernel` (0 = verify, 1 = realign, with the fused position ids
 * / mask in specdec_step, 2 = position ids / mask alone, 3 = batch gather,
 * 4 = write-back, 5 = stochastic verification, 6 = variable-length rollback,
 * 7 = the vocabulary scan of greedy verification alone, the first of its two
 * launches, 8 = the row statistics of stochastic verification alone, the
 * first of its four launches) and returns the totals since the last reset.
 * Launches recorded into a graph capture are not timed.
 */
#define SPECDEC_KERNEL_VERIFY 0
#define SPECDEC_KERNEL_REALIGN 1
#define SPECDEC_KERNEL_POSMASK 2
#define SPECDEC_KERNEL_GATHER 3
#define SPECDEC_KERNEL_WRITEBACK 4
#define SPECDEC_KERNEL_SAMPLE 5
#define SPECDEC_KERNEL_VARLEN 6
#define SPECDEC_KERNEL_VERIFY_SCAN 7
#define SPECDEC_KERNEL_SAMPLE_STATS 8
#define SPECDEC_TIMING_ALL 511
specdec_status_t specdec_timing_enable(int32_t kernel_mask);
specdec_status_t specdec_timing_reset(void);
specdec_status_t specdec_timing_query(int32_t kernel, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* SPECDEC_H */
