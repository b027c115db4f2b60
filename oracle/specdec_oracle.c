/*
 * Oracle for one step of batch speculative decoding under the EqSpec method:
 * greedy batch verification followed by "unpad-append-repad" realignment of a
 * left-padded contiguous KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, scalar CPU
 * definition that the HIP library is checked against.  It shares no code,
 * header, table or helper with the library; nothing in the product path may
 * link or call it.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.
 *
 * What it follows (arXiv 2510.22876):
 *   - BatchVerify, Algorithm 3 (Appendix "BatchVerify Algorithm Details"):
 *     predicted tokens are the argmax over the vocabulary, the first mismatch
 *     against the drafts gives the accepted prefix, and the bonus token is the
 *     target's prediction at the first mismatch.
 *   - Equation (1): the new batch width is the longest updated row,
 *     L' = max_j (c_j + a_j); Equation (2): per-row padding offset
 *     delta_i = (L' - L) - a_i; new padding p_i + delta_i.
 *   - Invariant I1 (rectangular alignment, p_i + c_i = L for every row) and
 *     invariant I2 (position ids are the running count of content tokens
 *     minus one, floored at zero; every content column carries the cached
 *     entry of its own token).
 *   - Section 3.1, paragraph "Unpad-Append-Repad" and Theorem B.1: realignment
 *     is a relocation; kept entries are moved unchanged, rejected entries are
 *     dropped, and the bonus token has no cache entry yet.
 *
 * Readings taken where the paper is silent or ambiguous (each is listed in
 * the design notes of the repository):
 *   - Cache state model.  Before the step, row i holds c_i = L - p_i cached
 *     entries in columns [p_i, L) of a width-L region, followed by the k+1
 *     entries the target just computed for the verify window
 *     [pending token, d_1 .. d_k] in columns [L, L+k+1).  The window's logit
 *     rows r = 0..k predict the token after window slot r.  The number of
 *     entries appended to the cache is a_i = (accepted drafts) + 1: the
 *     pending token plus each accepted draft; the bonus token becomes the new
 *     pending token.  In token terms this is the paper's a_i (accepted +
 *     bonus), so Eq. (1) and Eq. (2) apply unchanged with L counted in cache
 *     columns.
 *   - When every draft matches, Algorithm 3's argmax over the all-false
 *     mismatch vector would return 0; the accepted count is k instead and the
 *     bonus is the prediction after the last draft.
 *   - The bonus token is the prediction at window slot n_acc (0-based),
 *     independent of left padding.
 *   - Ties in the argmax go to the lowest index; -0.0 equals +0.0; a NaN
 *     ranks above every number and the first NaN wins.
 *   - Pad columns of the cache hold bf16 +0.0; position ids of pad columns
 *     are 0 (the max(0, .) of I2); the mask is 1 on content columns.
 *   - Position ids and the mask are emitted for columns [0, L'+k+1): the
 *     realigned cache plus the next verify window.
 *
 * Floating point: logits are widened exactly to double and compared there.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_BF16 = 1, OR_F16 = 2 };

enum {
  OR_OK = 0,
  OR_EINVAL = 1,   /* an argument is out of range */
  OR_ENOMEM = 2,
};

/* ---- exact widening of one logit to double -------------------------------- */

static double half_bits_to_double(uint16_t h) {
  int sign = h >> 15;
  int e = (h >> 10) & 0x1F;
  int m = h & 0x3FF;
  double v;
  if (e == 0) {
    v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
  } else if (e == 31) {
    v = m ? NAN : INFINITY;
  } else {
    v = ldexp((double)(m | 0x400), e - 25);    /* (1 + m/1024) * 2^(e-15) */
  }
  return sign ? -v : v;
}

static double logit_at(const void* base, int dtype, int64_t i) {
  if (dtype == OR_F32) {
    float f;
    memcpy(&f, (const char*)base + 4 * i, 4);
    return (double)f;
  }
  uint16_t h;
  memcpy(&h, (const char*)base + 2 * i, 2);
  if (dtype == OR_BF16) {
    uint32_t u = (uint32_t)h << 16;            /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
  }
  return half_bits_to_double(h);
}

int oracle_logit_bytes(int dtype) {
  return dtype == OR_F32 ? 4 : (dtype == OR_BF16 || dtype == OR_F16) ? 2 : 0;
}

/* Greedy prediction of one logit row (Algorithm 3: argmax over the
 * vocabulary).  Lowest index among equal maxima; the first NaN wins.
 * Returns -1 for an empty row or an unknown dtype. */
int64_t oracle_argmax(const void* row, int dtype, int64_t V) {
  if (V <= 0 || oracle_logit_bytes(dtype) == 0) return -1;
  int64_t best = 0;
  double best_v = logit_at(row, dtype, 0);
  if (isnan(best_v)) return 0;
  for (int64_t v = 1; v < V; ++v) {
    double x = logit_at(row, dtype, v);
    if (isnan(x)) return v;
    if (x > best_v) {           /* strict: an equal value later keeps the earlier index */
      best_v = x;
      best = v;
    }
  }
  return best;
}

/* ---- verification and the width / offset rule ---------------------------- */

/*
 * logits  [B][k+1][V] (dtype), row r of sequence i scores the token after
 *         verify-window slot r
 * draft   [B][k]      draft tokens d_1..d_k
 * pad_in  [B]         p_i, left padding before the step
 * W_in                width of the cache handed in, including the k+1 window
 *                     columns; L = W_in - (k+1)
 * outputs: tokens [B][k+1] (target predictions), n_acc [B] (accepted drafts,
 *          0..k), bonus [B], pad_out [B] (p_i + delta_i), *w_new (L')
 */
int oracle_verify(const void* logits, int dtype, const int32_t* draft, const int32_t* pad_in,
                  int32_t B, int32_t k, int64_t V, int32_t W_in,
                  int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                  int32_t* w_new) {
  int eb = oracle_logit_bytes(dtype);
  if (B < 0 || k < 0 || V <= 0 || eb == 0 || W_in < k + 1) return OR_EINVAL;
  const int32_t L = W_in - (k + 1);
  for (int32_t i = 0; i < B; ++i)
    if (pad_in[i] < 0 || pad_in[i] > L) return OR_EINVAL;

  /* Algorithm 3: pred_tokens <- argmax(logits, dim=vocab) */
  for (int32_t i = 0; i < B; ++i)
    for (int32_t r = 0; r <= k; ++r) {
      const char* row = (const char*)logits + ((int64_t)i * (k + 1) + r) * V * eb;
      tokens[(int64_t)i * (k + 1) + r] = (int32_t)oracle_argmax(row, dtype, V);
    }

  /* first mismatch j between pred_tokens and D; A[i] = D[i][:j];
   * bonus B[i] = prediction at the first mismatch (k when all match) */
  for (int32_t i = 0; i < B; ++i) {
    int32_t j = k;
    for (int32_t r = 0; r < k; ++r)
      if (draft[(int64_t)i * k + r] != tokens[(int64_t)i * (k + 1) + r]) {
        j = r;
        break;
      }
    n_acc[i] = j;
    if (bonus) bonus[i] = tokens[(int64_t)i * (k + 1) + j];
  }

  /* Eq. (1): L' = max_j (c_j + a_j), with c_j = L - p_j and a_j = n_acc + 1 */
  int32_t Lp = 0;
  for (int32_t i = 0; i < B; ++i) {
    int32_t c = L - pad_in[i];
    int32_t a = n_acc[i] + 1;
    if (c + a > Lp) Lp = c + a;
  }
  /* Eq. (2): delta_i = (L' - L) - a_i; new padding p_i + delta_i */
  for (int32_t i = 0; i < B; ++i) {
    int32_t a = n_acc[i] + 1;
    int32_t delta = (Lp - L) - a;
    pad_out[i] = pad_in[i] + delta;
  }
  *w_new = Lp;
  return OR_OK;
}

/* ---- KV realignment: unpad, append, repad ---------------------------------- */

/*
 * src  bf16 [n_layers][2][B][H][src_cap][D] (raw 16-bit patterns)
 * dst  bf16 [n_layers][2][B][H][dst_cap][D]; columns [0, w_new) of every row
 *      are written, columns beyond are left untouched
 * pad_in, n_acc [B]; w_new = L' from verification; W_in as in oracle_verify.
 *
 * For every (layer, K/V, row, head) span: unpad (take the c_i cached entries
 * in [p_i, L)), append (the first a_i = n_acc+1 window entries, columns
 * [L, L+a_i); the rest of the window belongs to rejected drafts and is
 * dropped), repad (write w_new - (c_i + a_i) zero columns, then the entries).
 * src and dst must not overlap.
 */
int oracle_realign_kv(const uint16_t* src, int64_t src_cap, uint16_t* dst, int64_t dst_cap,
                      int32_t n_layers, int32_t B, int32_t H, int32_t D, int32_t k,
                      int32_t W_in, const int32_t* pad_in, const int32_t* n_acc, int32_t w_new) {
  if (n_layers < 0 || B < 0 || H < 0 || D <= 0 || k < 0 || W_in < k + 1) return OR_EINVAL;
  if (src_cap < W_in || dst_cap < w_new || w_new < 0) return OR_EINVAL;
  const int32_t L = W_in - (k + 1);
  for (int32_t i = 0; i < B; ++i) {
    if (pad_in[i] < 0 || pad_in[i] > L || n_acc[i] < 0 || n_acc[i] > k) return OR_EINVAL;
    if ((L - pad_in[i]) + n_acc[i] + 1 > w_new) return OR_EINVAL;
  }
  uint16_t* row = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)(W_in > 0 ? W_in : 1) * (size_t)D);
  if (!row) return OR_ENOMEM;
  for (int32_t l = 0; l < n_layers; ++l)
    for (int32_t kv = 0; kv < 2; ++kv)
      for (int32_t i = 0; i < B; ++i)
        for (int32_t h = 0; h < H; ++h) {
          int64_t span = (((int64_t)l * 2 + kv) * B + i) * H + h;
          const uint16_t* s = src + span * src_cap * D;
          uint16_t* d = dst + span * dst_cap * D;
          int32_t c = L - pad_in[i];
          int32_t a = n_acc[i] + 1;
          int64_t n = 0;
          /* unpad: the cached content of the row */
          for (int32_t j = pad_in[i]; j < L; ++j, ++n)
            memcpy(row + n * D, s + (int64_t)j * D, sizeof(uint16_t) * D);
          /* append: entries of the pending token and the accepted drafts */
          for (int32_t j = L; j < L + a; ++j, ++n)
            memcpy(row + n * D, s + (int64_t)j * D, sizeof(uint16_t) * D);
          /* repad to the new width with fresh left padding */
          int32_t p_new = w_new - (c + a);
          for (int64_t j = 0; j < p_new; ++j)
            memset(d + j * D, 0, sizeof(uint16_t) * D);
          memcpy(d + (int64_t)p_new * D, row, sizeof(uint16_t) * (size_t)n * D);
        }
  free(row);
  return OR_OK;
}

/* ---- token row realignment (Alg. 1, phase 3) -------------------------------- */

/*
 * The token row S of each sequence before the step holds p_i pad tokens and
 * then c_i + 1 tokens: the c_i tokens whose entries are cached and the pending
 * token (its entry is computed by the verify forward), so its width is L + 1.
 * Phase 3 appends the accepted drafts and the bonus token (a_i = n_acc + 1
 * tokens: tokens[i][0..n_acc], the target's predictions, which equal the
 * accepted drafts) and repads every row to the new width L' + 1.
 *
 * s_in   int32 [B][s_in_stride], columns [0, L+1) read
 * s_out  int32 [B][s_out_stride], columns [0, L'+1) written
 * tokens int32 [B][k+1] from verification; pad_in, n_acc [B]; w_new = L'.
 * s_in and s_out must not overlap.
 */
int oracle_realign_tokens(const int32_t* s_in, int64_t s_in_stride, int32_t* s_out, int64_t s_out_stride,
                          const int32_t* tokens, const int32_t* pad_in, const int32_t* n_acc, int32_t w_new,
                          int32_t B, int32_t k, int32_t W_in, int32_t pad_id) {
  if (B < 0 || k < 0 || W_in < k + 1) return OR_EINVAL;
  const int32_t L = W_in - (k + 1);
  if (s_in_stride < (int64_t)L + 1 || s_out_stride < (int64_t)w_new + 1 || w_new < 0) return OR_EINVAL;
  int32_t* row = (int32_t*)malloc(sizeof(int32_t) * (size_t)(L + k + 2));
  if (!row) return OR_ENOMEM;
  for (int32_t i = 0; i < B; ++i) {
    if (pad_in[i] < 0 || pad_in[i] > L || n_acc[i] < 0 || n_acc[i] > k) {
      free(row);
      return OR_EINVAL;
    }
    const int32_t c = L - pad_in[i];
    const int32_t a = n_acc[i] + 1;
    if (c + a > w_new) {
      free(row);
      return OR_EINVAL;
    }
    int64_t n = 0;
    /* unpad: the sequence's own tokens, the pending token included */
    for (int32_t j = pad_in[i]; j <= L; ++j) row[n++] = s_in[(int64_t)i * s_in_stride + j];
    /* append: accepted drafts, then the bonus token */
    for (int32_t r = 0; r < a; ++r) row[n++] = tokens[(int64_t)i * (k + 1) + r];
    /* repad to width L' + 1 */
    const int64_t p_new = (int64_t)w_new + 1 - n;
    for (int64_t j = 0; j < p_new; ++j) s_out[(int64_t)i * s_out_stride + j] = pad_id;
    for (int64_t j = 0; j < n; ++j) s_out[(int64_t)i * s_out_stride + p_new + j] = row[j];
  }
  free(row);
  return OR_OK;
}

/* ---- EXSpec sequence pool: batch gather and write-back (Alg. 2) ------------- */

/*
 * The pool keeps every sequence unpadded: slot s holds len[s] cached entries
 * in cache columns [0, len[s]) of its spans and len[s] + 1 tokens (its cached
 * tokens and the pending token).
 *
 * Gather (Alg. 2, GetBatch): batch row i is slot slot[i], left-padded to the
 * batch width Lb: cache columns [0, Lb - len) hold +0.0 and [Lb - len, Lb) the
 * slot's entries; the token row holds Lb - len copies of pad_id, then the
 * slot's len + 1 tokens (width Lb + 1); pads[i] = Lb - len.  When every row
 * has the same length this is a plain concatenation (no padding).
 *
 * pool  bf16 [n_layers][2][N][H][pool_cap][D];  batch bf16 [n_layers][2][B][H][batch_cap][D]
 * pool_tok int32 [N][tok_stride];  batch_tok int32 [B][btok_stride]
 */
int oracle_gather_batch(const uint16_t* pool, int64_t pool_cap, int32_t N, const int32_t* pool_tok,
                        int64_t tok_stride, const int32_t* len, const int32_t* slot, int32_t B, int32_t Lb,
                        int32_t n_layers, int32_t H, int32_t D, uint16_t* batch, int64_t batch_cap,
                        int32_t* batch_tok, int64_t btok_stride, int32_t pad_id, int32_t* pads) {
  if (B < 0 || N < 0 || Lb < 0 || batch_cap < Lb || btok_stride < (int64_t)Lb + 1) return OR_EINVAL;
  for (int32_t i = 0; i < B; ++i) {
    if (slot[i] < 0 || slot[i] >= N) return OR_EINVAL;
    const int32_t n = len[slot[i]];
    if (n < 0 || n > Lb || n > pool_cap || (int64_t)n + 1 > tok_stride) return OR_EINVAL;
  }
  for (int32_t i = 0; i < B; ++i) {
    const int32_t n = len[slot[i]];
    const int32_t p = Lb - n;
    pads[i] = p;
    for (int32_t l = 0; l < n_layers; ++l)
      for (int32_t kv = 0; kv < 2; ++kv)
        for (int32_t h = 0; h < H; ++h) {
          const uint16_t* s = pool + ((((int64_t)l * 2 + kv) * N + slot[i]) * H + h) * pool_cap * D;
          uint16_t* d = batch + ((((int64_t)l * 2 + kv) * B + i) * H + h) * batch_cap * D;
          for (int64_t j = 0; j < p; ++j) memset(d + j * D, 0, sizeof(uint16_t) * D);
          memcpy(d + (int64_t)p * D, s, sizeof(uint16_t) * (size_t)n * D);
        }
    for (int32_t j = 0; j < p; ++j) batch_tok[(int64_t)i * btok_stride + j] = pad_id;
    for (int32_t j = 0; j <= n; ++j)
      batch_tok[(int64_t)i * btok_stride + p + j] = pool_tok[(int64_t)slot[i] * tok_stride + j];
  }
  return OR_OK;
}

/*
 * Write-back (Alg. 2, Phase 4): after verification of a batch formed by
 * gather (rows end at column Lb, row i has pads[i] columns of padding, the
 * verify window occupies [Lb, Lb + k + 1)), for every row i:
 *   Pool[slot] <- Pool[slot] + A[i] + B[i]: the slot's token list gains the
 *     accepted drafts and the bonus (tokens[i][0..n_acc[i]]);
 *   Pool.KV[slot] <- KV[i]: the slot's cache becomes the row's cache,
 *     unpadded and cut after the accepted entries: batch columns
 *     [pads[i], Lb + n_acc[i] + 1) -> slot columns [0, len + n_acc[i] + 1);
 *   len[slot] grows by n_acc[i] + 1.
 * The row must mirror its slot (len[slot] == Lb - pads[i]); slots must be
 * distinct.  When batch_tok is not NULL the batch's own token row (width
 * Lb + 1) also gains the n_acc[i] + 1 tokens at columns [Lb + 1, Lb + n_acc[i]
 * + 2): the step's append to S that a batch kept for the next step needs.
 */
int oracle_scatter_accepted(const uint16_t* batch, int64_t batch_cap, int32_t B, const int32_t* pads,
                            const int32_t* tokens, int32_t k, const int32_t* n_acc, const int32_t* slot, int32_t Lb,
                            int32_t n_layers, int32_t H, int32_t D, uint16_t* pool, int64_t pool_cap, int32_t N,
                            int32_t* pool_tok, int64_t tok_stride, int32_t* len, int32_t* batch_tok,
                            int64_t btok_stride) {
  if (B < 0 || N < 0 || k < 0 || Lb < 0 || batch_cap < (int64_t)Lb + k + 1) return OR_EINVAL;
  if (batch_tok && btok_stride < (int64_t)Lb + k + 2) return OR_EINVAL;
  for (int32_t i = 0; i < B; ++i) {
    if (slot[i] < 0 || slot[i] >= N || n_acc[i] < 0 || n_acc[i] > k) return OR_EINVAL;
    if (pads[i] < 0 || pads[i] > Lb || len[slot[i]] != Lb - pads[i]) return OR_EINVAL;
    for (int32_t q = 0; q < i; ++q)
      if (slot[q] == slot[i]) return OR_EINVAL;
    const int64_t grown = (int64_t)len[slot[i]] + n_acc[i] + 1;
    if (grown > pool_cap || grown + 1 > tok_stride) return OR_EINVAL;
  }
  for (int32_t i = 0; i < B; ++i) {
    const int32_t a = n_acc[i] + 1;
    const int32_t n = Lb - pads[i];
    for (int32_t l = 0; l < n_layers; ++l)
      for (int32_t kv = 0; kv < 2; ++kv)
        for (int32_t h = 0; h < H; ++h) {
          const uint16_t* s = batch + ((((int64_t)l * 2 + kv) * B + i) * H + h) * batch_cap * D;
          uint16_t* d = pool + ((((int64_t)l * 2 + kv) * N + slot[i]) * H + h) * pool_cap * D;
          memcpy(d, s + (int64_t)pads[i] * D, sizeof(uint16_t) * (size_t)(n + a) * D);
        }
    int32_t* trow = pool_tok + (int64_t)slot[i] * tok_stride;
    for (int32_t r = 0; r < a; ++r) trow[n + 1 + r] = tokens[(int64_t)i * (k + 1) + r];
    if (batch_tok)
      for (int32_t r = 0; r < a; ++r) batch_tok[(int64_t)i * btok_stride + Lb + 1 + r] = tokens[(int64_t)i * (k + 1) + r];
    len[slot[i]] = n + a;
  }
  return OR_OK;
}

/* ---- position ids and attention mask (I2) ---------------------------------- */

/*
 * For columns j in [0, w_new + k + 1): mask[i][j] = 1 on content (j >= pad_out[i]),
 * pos[i][j] = max(0, (number of content columns q <= j) - 1).
 * pos, mask are [B][pm_cap].
 */
int oracle_posmask(const int32_t* pad_out, int32_t w_new, int32_t B, int32_t k,
                   int64_t* pos, uint8_t* mask, int64_t pm_cap) {
  if (B < 0 || k < 0 || w_new < 0 || pm_cap < (int64_t)w_new + k + 1) return OR_EINVAL;
  const int64_t width = (int64_t)w_new + k + 1;
  for (int32_t i = 0; i < B; ++i) {
    if (pad_out[i] < 0 || pad_out[i] > w_new) return OR_EINVAL;
    int64_t count = 0;
    for (int64_t j = 0; j < width; ++j) {
      uint8_t m = (j >= pad_out[i]) ? 1 : 0;
      mask[(int64_t)i * pm_cap + j] = m;
      count += m;
      pos[(int64_t)i * pm_cap + j] = count - 1 > 0 ? count - 1 : 0;
    }
  }
  return OR_OK;
}

/* ---- stochastic verification (temperature T > 0) --------------------------- */

/*
 * At T > 0, output equivalence means the emitted tokens follow the target
 * model's distribution (Section 2, the equivalence requirement), which the
 * speculative-sampling rule the paper builds on guarantees (Chen et al.,
 * 2023, "Accelerating large language model decoding with speculative
 * sampling"; Leviathan et al., 2023).  With target distributions
 * p_r = softmax(logits[i][r] / T) and draft distributions
 * q_r = softmax(draft_logits[i][r] / T):
 *   - draft x_r = draft[i][r] is accepted iff u_accept[i][r] * q_r(x_r) <
 *     p_r(x_r), i.e. with probability min(1, p_r(x_r) / q_r(x_r));
 *   - at the first rejected slot r, the correction token is sampled from the
 *     residual distribution proportional to max(0, p_r - q_r);
 *   - when all k drafts are accepted, the bonus token is sampled from p_k.
 * Sampling uses one uniform per row, u_sample[i], by inversion: the smallest
 * index j whose cumulative weight exceeds u_sample[i] times the total.
 * Readings: one temperature for target and draft; a residual with zero mass
 * (only possible when p_r(x_r) = q_r(x_r) = 0) falls back to p_r; a draft id
 * outside [0, V) has probability 0 under both and is rejected; the accepted
 * drafts and then the sampled token form tokens[i][0 .. n_acc] (later entries
 * are -1); the width and paddings follow Eq. (1) and Eq. (2) as in greedy
 * verification.  Everything is computed in double.  Logits must be finite or
 * -inf, with a finite maximum per row.
 */

/* p = softmax(row / T), in double, with the row's maximum subtracted */
static void softmax_row(const void* row, int dtype, int64_t V, double T, double* p) {
  double m = -INFINITY;
  for (int64_t v = 0; v < V; ++v) {
    double x = logit_at(row, dtype, v);
    if (x > m) m = x;
  }
  double z = 0.0;
  for (int64_t v = 0; v < V; ++v) {
    p[v] = exp((logit_at(row, dtype, v) - m) / T);
    z += p[v];
  }
  for (int64_t v = 0; v < V; ++v) p[v] /= z;
}

/* inversion: the smallest j with w_0 + .. + w_j > u * (w_0 + .. + w_{V-1});
 * the last index of positive weight when rounding leaves none; -1 if all are 0 */
static int64_t sample_by_inversion(const double* w, int64_t V, double u) {
  double total = 0.0;
  for (int64_t v = 0; v < V; ++v) total += w[v];
  const double target = u * total;
  double c = 0.0;
  int64_t last = -1;
  for (int64_t v = 0; v < V; ++v) {
    if (w[v] > 0.0) last = v;
    c += w[v];
    if (c > target) return v;
  }
  return last;
}

int oracle_verify_sample(const void* logits, const void* draft_logits, int dtype, const int32_t* draft,
                         const int32_t* pad_in, const float* u_accept, const float* u_sample,
                         double temperature, int32_t B, int32_t k, int64_t V, int32_t W_in,
                         int32_t* tokens, int32_t* n_acc, int32_t* bonus, int32_t* pad_out,
                         int32_t* w_new) {
  int eb = oracle_logit_bytes(dtype);
  if (B < 0 || k < 0 || V <= 0 || eb == 0 || W_in < k + 1) return OR_EINVAL;
  if (!(temperature > 0.0) || !isfinite(temperature)) return OR_EINVAL;
  const int32_t L = W_in - (k + 1);
  for (int32_t i = 0; i < B; ++i) {
    if (pad_in[i] < 0 || pad_in[i] > L) return OR_EINVAL;
    if (!(u_sample[i] >= 0.0f && u_sample[i] < 1.0f)) return OR_EINVAL;
    for (int32_t r = 0; r < k; ++r)
      if (!(u_accept[(int64_t)i * k + r] >= 0.0f && u_accept[(int64_t)i * k + r] < 1.0f)) return OR_EINVAL;
  }
  double* p = (double*)malloc(sizeof(double) * (size_t)V);
  double* q = (double*)malloc(sizeof(double) * (size_t)V);
  double* w = (double*)malloc(sizeof(double) * (size_t)V);
  if (!p || !q || !w) {
    free(p); free(q); free(w);
    return OR_ENOMEM;
  }
  for (int32_t i = 0; i < B; ++i) {
    int32_t acc = k;
    int64_t x_out = -1;
    for (int32_t r = 0; r < k; ++r) {
      softmax_row((const char*)logits + ((int64_t)i * (k + 1) + r) * V * eb, dtype, V, temperature, p);
      softmax_row((const char*)draft_logits + ((int64_t)i * k + r) * V * eb, dtype, V, temperature, q);
      const int32_t x = draft[(int64_t)i * k + r];
      const double px = (x >= 0 && x < V) ? p[x] : 0.0;
      const double qx = (x >= 0 && x < V) ? q[x] : 0.0;
      if ((double)u_accept[(int64_t)i * k + r] * qx < px) continue;   /* accepted */
      acc = r;                                                           /* rejected: residual */
      for (int64_t v = 0; v < V; ++v) w[v] = p[v] > q[v] ? p[v] - q[v] : 0.0;
      x_out = sample_by_inversion(w, V, (double)u_sample[i]);
      if (x_out < 0) x_out = sample_by_inversion(p, V, (double)u_sample[i]);
      break;
    }
    if (acc == k) {                                                      /* all accepted: bonus from p_k */
      softmax_row((const char*)logits + ((int64_t)i * (k + 1) + k) * V * eb, dtype, V, temperature, p);
      x_out = sample_by_inversion(p, V, (double)u_sample[i]);
    }
    n_acc[i] = acc;
    for (int32_t r = 0; r <= k; ++r)
      tokens[(int64_t)i * (k + 1) + r] = r < acc ? draft[(int64_t)i * k + r] : (r == acc ? (int32_t)x_out : -1);
    if (bonus) bonus[i] = (int32_t)x_out;
  }
  free(p); free(q); free(w);
  /* Eq. (1) and Eq. (2) */
  int32_t Lp = 0;
  for (int32_t i = 0; i < B; ++i)
    if ((L - pad_in[i]) + n_acc[i] + 1 > Lp) Lp = (L - pad_in[i]) + n_acc[i] + 1;
  for (int32_t i = 0; i < B; ++i) pad_out[i] = pad_in[i] + ((Lp - L) - (n_acc[i] + 1));
  *w_new = Lp;
  return OR_OK;
}

/* ---- rollback (Family A) and variable-length rollback (Family B) ------------ */

/*
 * Rollback (Section 2, "Family A: contiguous layout"): every row is truncated
 * to the batch-minimum accepted count m = min_i n_acc[i], so every row appends
 * the same a = m + 1 cache entries and the same tokens[i][0 .. m] (for a row
 * that accepted more, tokens[i][m] is the target's prediction at slot m, equal
 * to its draft there).  The width and paddings then follow Eq. (1) and
 * Eq. (2) with a_i = m + 1 for every row; all offsets are equal (zero when the
 * minimum input padding is 0, Corollary B.4), so no cached entry moves.
 * Verified tokens beyond m are discarded.
 */
int oracle_rollback(const int32_t* tokens, const int32_t* n_acc, const int32_t* pad_in, int32_t B, int32_t k,
                    int32_t W_in, int32_t* n_acc_out, int32_t* bonus_out, int32_t* pad_out, int32_t* w_new) {
  if (B < 0 || k < 0 || W_in < k + 1) return OR_EINVAL;
  const int32_t L = W_in - (k + 1);
  int32_t m = k;
  for (int32_t i = 0; i < B; ++i) {
    if (pad_in[i] < 0 || pad_in[i] > L || n_acc[i] < 0 || n_acc[i] > k) return OR_EINVAL;
    if (n_acc[i] < m) m = n_acc[i];
  }
  int32_t Lp = 0;
  for (int32_t i = 0; i < B; ++i) {
    n_acc_out[i] = m;
    bonus_out[i] = tokens[(int64_t)i * (k + 1) + m];
    if ((L - pad_in[i]) + m + 1 > Lp) Lp = (L - pad_in[i]) + m + 1;   /* Eq. (1) */
  }
  for (int32_t i = 0; i < B; ++i) pad_out[i] = pad_in[i] + ((Lp - L) - (m + 1));   /* Eq. (2) */
  *w_new = B > 0 ? Lp : 0;
  return OR_OK;
}

/*
 * Variable-length rollback (Section 2, "Family B: variable-length layout"):
 * the cache is a flat buffer per (layer, K/V), [T][H][D], sequence i holding
 * rows [cu_in[i], cu_in[i+1]): its cached entries followed by its k+1 verify
 * window entries.  I1 does not arise; I2 requires the rejected entries to be
 * rolled back: sequence i keeps its first len_i - (k - n_acc[i]) rows (the
 * window entries of the pending token and the accepted drafts) and the
 * buffer is compacted, cu_out being the running sum of the kept lengths.
 * Position ids are each kept row's index within its sequence.  Rows of the
 * output beyond cu_out[B] are left as they are.
 *   src, dst  bf16 bits [n_layers][2][T_cap][H][D] (dst separate from src)
 *   pos       int64 [T_cap]: positions for rows [0, cu_out[B])
 */
int oracle_varlen_rollback(const uint16_t* src, uint16_t* dst, int64_t T_cap, int32_t n_layers, int32_t H, int32_t D,
                           const int32_t* cu_in, const int32_t* n_acc, int32_t B, int32_t k, int32_t* cu_out,
                           int64_t* pos) {
  if (B < 0 || k < 0 || n_layers < 0 || H < 0 || D <= 0 || T_cap < 0) return OR_EINVAL;
  if (cu_in[0] < 0) return OR_EINVAL;
  for (int32_t i = 0; i < B; ++i) {
    const int64_t len = (int64_t)cu_in[i + 1] - cu_in[i];
    if (len < k + 1 || cu_in[i + 1] > T_cap || n_acc[i] < 0 || n_acc[i] > k) return OR_EINVAL;
  }
  const int64_t row = (int64_t)H * D;
  cu_out[0] = 0;
  for (int32_t i = 0; i < B; ++i) {
    const int64_t keep = (int64_t)cu_in[i + 1] - cu_in[i] - (k - n_acc[i]);
    cu_out[i + 1] = cu_out[i] + (int32_t)keep;
    for (int32_t l = 0; l < n_layers; ++l)
      for (int32_t kv = 0; kv < 2; ++kv) {
        const uint16_t* s = src + ((int64_t)l * 2 + kv) * T_cap * row + (int64_t)cu_in[i] * row;
        uint16_t* d = dst + ((int64_t)l * 2 + kv) * T_cap * row + (int64_t)cu_out[i] * row;
        memcpy(d, s, sizeof(uint16_t) * (size_t)(keep * row));
      }
    for (int64_t t = 0; t < keep; ++t) pos[cu_out[i] + t] = t;
  }
  return OR_OK;
}
