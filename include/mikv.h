/*
 * mikv.h -- C ABI of libmikv.so: the decode hot path of MiKV
 * ("No Token Left Behind: Reliable KV Cache Compression via Importance-Aware
 * Mixed Precision Quantization", arXiv 2402.18096) for AMD MI355X (gfx950).
 *
 * A MiKV cache keeps, per (sequence, KV head), the tokens ranked important
 * by accumulated attention at high precision (fp16, INT8 or INT4: the
 * "importance cache") and every other token at low precision (INT4/INT3/INT2,
 * per-token grouped asymmetric: the "retained cache") instead of evicting it
 * (Section 3, Fig. 3).  Because attention after RoPE is permutation
 * invariant, the two precisions are stored as two separate pools (Section
 * 3.4); a token's position travels with it in a position array.
 *
 * Conventions shared by every entry point
 *  - All pointers named in a mikv_cache and every array argument are DEVICE
 *    pointers unless stated otherwise.  The caller allocates everything; the
 *    library allocates no memory and keeps no state between calls apart from
 *    its loaded code objects (which hold the device scratch array of
 *    mikv_decode_step_noalloc).
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  Results are valid once the stream has synchronised.  Calls on
 *    distinct buffers are thread safe; overlapping calls on one cache race.
 *  - fp16 data is passed as uint16_t bit patterns (IEEE binary16).
 *  - Return value: MIKV_OK or an error code.  Argument validation happens on
 *    the host before any launch; on a validation error nothing is launched
 *    and nothing is written.  mikv_last_error() gives a message for the
 *    calling thread's last error.  No call throws, aborts or prints.
 *  - Overflow of a pool capacity can only be detected on the device (the
 *    host does not know the pool fill levels); kernels then skip the
 *    offending writes (never writing out of bounds) and OR a MIKV_DEVERR_*
 *    bit into the cache's `status` word, which the caller may read.
 *  - NaN or infinite inputs give unspecified (but in-bounds) results.
 *  - head_dim must be 128.
 */
#ifndef MIKV_H
#define MIKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum mikv_status {
  MIKV_OK = 0,
  MIKV_ERR_INVALID_ARG = 1, /* null pointer, bad shape or inconsistent sizes */
  MIKV_ERR_UNSUPPORTED = 2, /* head_dim != 128, unsupported bit width / group / GQA group */
  MIKV_ERR_CAPACITY = 3,    /* host-detectable capacity overflow (length > max_len, workspace too small) */
  MIKV_ERR_HIP = 4          /* a HIP launch failed (hipGetLastError) */
};

/* Bits of mikv_cache.status, set on the device. */
enum mikv_device_error {
  MIKV_DEVERR_HI_FULL = 1, /* importance pool overflow: token not stored */
  MIKV_DEVERR_LO_FULL = 2, /* retained pool overflow: token not stored */
  MIKV_DEVERR_KEY_BLOCK = 4 /* key_block 64: a token for the retained pool whose key block is not
                               complete, or a completed block with a key outside the importance
                               pool (token or block parameters not stored) */
};

/* Flags of mikv_decode_attention. */
enum mikv_attention_flags {
  /* Also add the step's probabilities of importance-pool tokens to their
   * scores (the mikv_importance_update of the same step, fused). */
  MIKV_ATTN_ACCUMULATE = 1
};

/*
 * The cache of B sequences x Hkv KV heads.  NH = B * Hkv independent heads;
 * head index h = b * Hkv + kv_head.  Every pool array is [NH, cap, ...]
 * row-major.
 *
 * Importance pool (high precision, Section 3.3):
 *   hi_bits == 16: hi_k, hi_v are fp16 [NH, cap_hi, 128]; hi_kp, hi_vp unused.
 *   hi_bits == 8 : hi_k, hi_v are uint8 codes [NH, cap_hi, 128];
 *                  hi_kp, hi_vp are fp16 (alpha, beta) pairs [NH, cap_hi, 128/group, 2].
 *   hi_bits == 4 : the INT4 importance cache of Table 3 (with lo_bits 2 or 0):
 *                  hi_k, hi_v are packed codes [NH, cap_hi, 64] (LSB first, as
 *                  the retained pool's); hi_kp, hi_vp as for INT8.
 *   hi_pos  [NH, cap_hi] int32: token position held by each slot.
 *   hi_acc  [NH, cap_hi] fp32 : the token's accumulated attention (H2O score).
 *   n_hi    [NH] int32        : occupied slots (slots [0, n_hi) are valid).
 * Retained pool (low precision, Section 3.1):
 *   lo_k, lo_v   uint8 packed codes [NH, cap_lo, 128 * lo_bits / 8];
 *   lo_kp, lo_vp fp16 (alpha, beta) pairs [NH, cap_lo, 128/group, 2];
 *   lo_pos [NH, cap_lo] int32; n_lo [NH] int32.
 * lo_bits == 0 selects the paper's eviction baseline (H2O, the cache with
 *   0-bit retained tokens of Section 4 / Table 1): there is no retained
 *   pool, a token left out of the importance pool at prefill or demoted by
 *   the re-rank is dropped, and attention covers the importance pool only.
 *   lo_k, lo_v, lo_kp, lo_vp and lo_pos are then unused (may be NULL),
 *   cap_lo is ignored, n_lo (still required) stays as the caller set it,
 *   probs_lo is not written, and map 0 means "evicted".
 * Codes: Eq. 1 per token and per group of `group` contiguous channels, packed
 * least-significant-bits first (channel c at byte c*N/8, bit (c*N)%8).
 * Exception: 2-bit retained values of a cache shared by two or more query
 *   heads (q_heads >= 2 * kv_heads) are stored in tiles of 32 slots (cap_lo a
 *   multiple of 32) for the matrix cores: byte q (0..31) of slot s holds
 *   channels q, q+32, q+64, q+96 at bits 0-1, 2-3, 4-5, 6-7 and sits at
 *   (s/32)*1024 + 16*(16*((s%32)/8) + q%16) + 8*(q/16) + s%8 of the head's
 *   array (same size as the token-major one).
 * Keys are stored balanced (Eq. 3) when a balancer is in use.
 * map [NH, max_len] uint8 (nullable): 1 = position in the importance pool,
 *   0 = retained pool; maintained by mikv_quantize_kv and mikv_select_topk.
 * status: one device int32 (required), see mikv_device_error.
 * Retained-pool tokens carry no score: they are never promoted again, so
 * their score would never be read.
 *
 * Per-channel key quantization (Appendix C, Table 6): key_block 64 quantizes
 * the retained pool's keys per channel over blocks of 64 consecutive
 * positions instead of per token (values stay per token).  The parameters of
 * block b = positions [64 b, 64 b + 64) are Eq. 1 over the block's 64 keys,
 * channel by channel, taken when the block is complete (from the keys given
 * to mikv_quantize_kv, or from the importance pool when the block completes
 * during decoding: with a window of at least 64 positions every key of an
 * incomplete block is still there):
 *   lo_kb fp16 (alpha, beta) pairs [NH, max_len / 64, 128, 2];
 * a retained key's codes (lo_k, packed as before) are Eq. 1 of its fp16 key
 * with its block's parameters of each channel; lo_kp is unused (may be
 * NULL).  Requires hi_bits 16, lo_bits 2, 3 or 4, one query head per KV
 * head, no balancer, and a window of at least 64 in the re-rank.
 */
typedef struct mikv_cache {
  int32_t batch;
  int32_t q_heads;
  int32_t kv_heads;   /* q_heads % kv_heads == 0; q_heads / kv_heads in {1,2,4,8} */
  int32_t head_dim;   /* 128 */
  int32_t group;      /* quantization group size: 32, 64 or 128 channels */
  int32_t hi_bits;    /* 16 (fp16), 8 (INT8) or 4 (INT4, with lo_bits 2 or 0) */
  int32_t lo_bits;    /* 2, 3, 4 or 8; 0 = evict instead of retaining (see above) */
  int32_t cap_hi;     /* importance-pool slots per head */
  int32_t cap_lo;     /* retained-pool slots per head (ignored when lo_bits is 0) */
  int32_t max_len;    /* positions per head (length of map rows) */
  void *hi_k, *hi_v;
  uint16_t *hi_kp, *hi_vp;
  int32_t *hi_pos;
  float *hi_acc;
  int32_t *n_hi;
  uint8_t *lo_k, *lo_v;
  uint16_t *lo_kp, *lo_vp;
  int32_t *lo_pos;
  int32_t *n_lo;
  uint8_t *map;
  int32_t *status;
  int32_t key_block;  /* 0: retained keys per token and channel group; 64: per channel and block of 64 positions */
  uint16_t *lo_kb;    /* key_block 64: per-block key parameters (see above); else unused */
} mikv_cache;

/* Message describing the calling thread's last error ("" if none). */
const char *mikv_last_error(void);

/*
 * Channel balancer, Section 3.2, Eq. 2:
 *   balance[b, h, c] = sqrt( max_{t, i in group(h)} |q[b, i, t, c]| / max_t |k[b, h, t, c]| )
 * over the prefill prompt, in fp32 (correctly rounded divide and square
 * root); 1 where either maximum is 0.
 *   q_prefill fp16 [B, Hq, T, 128]; k_prefill fp16 [B, Hkv, T, 128], both
 *             16-byte aligned;
 *   balance   fp32 [B, Hkv, 128] (output);
 *   workspace device bytes, at least mikv_balance_workspace_size(B, Hkv, T).
 * Errors: INVALID_ARG for null or misaligned pointers, T < 1, Hq % Hkv != 0;
 * UNSUPPORTED for head_dim != 128; CAPACITY for a too-small workspace.
 */
size_t mikv_balance_workspace_size(int32_t batch, int32_t kv_heads, int32_t tokens);
int mikv_balance_channels(const uint16_t *q_prefill, const uint16_t *k_prefill, int32_t batch,
                          int32_t q_heads, int32_t kv_heads, int32_t tokens, int32_t head_dim,
                          float *balance, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Importance scores of the prompt (the H2O accumulated attention at the end
 * of prefill that ranks tokens for the first selection, Section 3.1 and the
 * H2O policy of Section 4.1): with causal softmax attention over the prompt,
 *   scores[b, h, j] = sum_{g in group(h)} sum_{i = j}^{T-1} softmax_i(scale * q[b, g, i] . k[b, h, :])_j
 * where group(h) are the Hq / Hkv query heads sharing KV head h.  Logits are
 * fp16 x fp16 products accumulated in fp32 on the matrix cores; the sums
 * are fp32 (summation order: per query head, query rows in ascending order,
 * then the heads of the group), so results are reproducible run to run but
 * not bit-identical to another summation order.
 *   q_prefill fp16 [B, Hq, T, 128]; k_prefill fp16 [B, Hkv, T, 128], both
 *             16-byte aligned (the prompt's keys as computed, before any
 *             balancing or quantization: balancing leaves q . k unchanged);
 *   scale     softmax scale (1/sqrt(128) for the paper's models), > 0;
 *   scores    fp32 [B, Hkv, T] (output), the `scores` argument of
 *             mikv_select_prefill and the score_init of mikv_quantize_kv;
 *   workspace device bytes, at least mikv_prefill_importance_workspace_size(B, Hq, T)
 *             (per-query softmax statistics).
 * Errors: INVALID_ARG for null or misaligned pointers, T < 1, Hq % Hkv != 0,
 * scale <= 0; UNSUPPORTED for head_dim != 128 or Hq / Hkv not in {1,2,4,8};
 * CAPACITY for a too-small workspace.
 */
size_t mikv_prefill_importance_workspace_size(int32_t batch, int32_t q_heads, int32_t tokens);
int mikv_prefill_importance(const uint16_t *q_prefill, const uint16_t *k_prefill, int32_t batch,
                            int32_t q_heads, int32_t kv_heads, int32_t tokens, int32_t head_dim, float scale,
                            float *scores, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Raw per-token grouped asymmetric quantizer, Section 3.1, Eq. 1, on rows of
 * 128 channels (for unit use and testing):
 *   x_c   = fp32(x[r, c]) * balance[r / rows_per_balance, c]   (balance nullable: x_c = fp32(x))
 *   alpha = fp16((max x - min x) / (2^bits - 1)), beta = fp16(min x) per group,
 *   code  = clamp(rint((x - beta) / alpha), 0, 2^bits - 1)  (all codes 0 if alpha == 0)
 * with fp32 arithmetic, round half to even, a correctly rounded divide and
 * the stored fp16 alpha and beta used for encoding.
 *   x      fp16 [rows, 128];   balance fp32 [rows / rows_per_balance, 128] or NULL;
 *   codes  uint8 [rows, 128 * bits / 8] (packed, LSB first);
 *   params fp16 (alpha, beta) pairs [rows, 128 / group, 2].
 * bits in {2, 3, 4, 8} (3-bit codes straddle bytes); group in {32, 64, 128}.  rows == 0 is a no-op (pointers may
 * then be NULL).
 */
int mikv_quantize_rows(const uint16_t *x, int64_t rows, int32_t head_dim, const float *balance,
                       int32_t rows_per_balance, int32_t bits, int32_t group, uint8_t *codes,
                       uint16_t *params, void *stream);

/*
 * Place n consecutive tokens, positions pos0 .. pos0+n-1, of every head into
 * the cache (prefill: the cache generated en masse, Section 2.1; decode: the
 * new token's key/value added each generation step).
 *   k, v       fp16 [B, Hkv, n, 128];
 *   balance    fp32 [B, Hkv, 128] or NULL (Eq. 3: keys are multiplied by it
 *              before quantization or fp16 storage; values are not balanced);
 *   hi_mask    uint8 [B, Hkv, n] or NULL (NULL: every token to the importance
 *              pool, as for a newly generated token);
 *   score_init fp32 [B, Hkv, n] or NULL: initial score of tokens entering the
 *              importance pool (NULL: 0, a new token's score).
 * Tokens are appended to their pool after the occupied slots, in position
 * order; hi_pos/lo_pos, n_hi/n_lo, hi_acc and map are updated.  Importance
 * tokens are stored as fp16 (hi_bits 16: fp16 of the fp32 balanced key) or
 * INT8/INT4 codes, retained tokens as lo_bits codes (dropped when lo_bits is
 * 0).
 *   workspace: at least mikv_quantize_workspace_size(c, n) bytes (0 when
 *   hi_mask is NULL).
 * Errors: INVALID_ARG (null pointers, n < 1, pos0 < 0), CAPACITY (pos0 + n >
 * max_len, workspace too small); pool overflow sets MIKV_DEVERR_* bits.
 */
size_t mikv_quantize_workspace_size(const mikv_cache *c, int32_t n);
int mikv_quantize_kv(const mikv_cache *c, const uint16_t *k, const uint16_t *v, const float *balance,
                     int32_t pos0, int32_t n, const uint8_t *hi_mask, const float *score_init,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * Decode-step attention over the mixed-precision cache, Section 3.4 and
 * Fig. 3 (left): K and V are dequantized on the fly (Eq. 1, alpha*code+beta,
 * or the fp16 value), the query stays floating point (q / balance, Eq. 4):
 *   s_j = (q_hat . k_j) * scale over every token j of both pools,
 *   p   = softmax(s),   out = sum_j p_j v_j,
 * accumulated in fp32, split over the sequence (split-K) and merged exactly.
 *   length    tokens per head currently in the cache (host-known bound on
 *             n_hi + n_lo; sizes the launch);
 *   q         fp16 [B, Hq, 128];  balance fp32 [B, Hkv, 128] or NULL;
 *   out       fp32 [B, Hq, 128];
 *   probs_hi  fp32 [B, Hq, cap_hi] or NULL: probabilities of importance-pool
 *             tokens, in slot order (entry [b, i, s] belongs to hi_pos[b*Hkv + i/G, s]);
 *   probs_lo  fp32 [B, Hq, cap_lo] or NULL: the same for the retained pool;
 *   flags     MIKV_ATTN_ACCUMULATE: also hi_acc[s] += sum over the group's
 *             query heads of probs_hi (left to right in head order, then one
 *             fp32 add) -- the importance update of this step, fused;
 *   workspace at least mikv_decode_workspace_size(c, length) bytes.
 * The call runs two phases that may also be launched separately:
 * _partial (per-chunk scores, softmax partials and value sums) and
 * _finalize (merge, probabilities, optional score update); both take the
 * same arguments and must see the same ones.
 * Errors: INVALID_ARG, UNSUPPORTED, CAPACITY (length > max_len, workspace).
 */
size_t mikv_decode_workspace_size(const mikv_cache *c, int32_t length);
int mikv_decode_attention(const mikv_cache *c, int32_t length, const uint16_t *q,
                          const float *balance, float scale, float *out, float *probs_hi,
                          float *probs_lo, int32_t flags, void *workspace, size_t workspace_bytes,
                          void *stream);
int mikv_decode_attention_partial(const mikv_cache *c, int32_t length, const uint16_t *q,
                                  const float *balance, float scale, float *out, float *probs_hi,
                                  float *probs_lo, int32_t flags, void *workspace,
                                  size_t workspace_bytes, void *stream);
int mikv_decode_attention_finalize(const mikv_cache *c, int32_t length, const uint16_t *q,
                                   const float *balance, float scale, float *out, float *probs_hi,
                                   float *probs_lo, int32_t flags, void *workspace,
                                   size_t workspace_bytes, void *stream);

/*
 * The attention's probabilities by token position (the softmax over the
 * sequence of Section 3.4 / Fig. 3, as the slot-ordered outputs of
 * mikv_decode_attention are laid out by the pools' position maps):
 *   probs[b, i, hi_pos[h, s]] = probs_hi[b, i, s]  for s < n_hi[h],
 *   probs[b, i, lo_pos[h, s]] = probs_lo[b, i, s]  for s < n_lo[h],
 * h = b*Hkv + i/G, and 0 for every other position below `length` (tokens
 * an evicting cache dropped).
 *   probs_hi, probs_lo  as written by mikv_decode_attention (probs_lo may be
 *                       NULL only for an evicting cache);
 *   probs               fp32 [B, Hq, length], written whole.
 * The slot maps must be those the attention saw: call it after
 * mikv_decode_attention and before mikv_select_topk moves slots (the fused
 * mikv_decode_step re-ranks in the same launch, so its outputs cannot be
 * remapped afterwards).
 * Errors: INVALID_ARG (NULL pointers, length < 1), CAPACITY (length >
 * max_len).
 */
int mikv_probs_by_position(const mikv_cache *c, int32_t length, const float *probs_hi, const float *probs_lo,
                           float *probs, void *stream);

/*
 * Importance update (the heavy-hitter accumulated attention policy MiKV
 * adopts, Sections 3.1 and 4.1): for every occupied importance-pool slot s,
 *   hi_acc[h, s] += ((probs_hi[b, hG, s] + probs_hi[b, hG+1, s]) + ...)
 * summing the G query heads of the KV group left to right in fp32, then one
 * fp32 add.  probs_hi as written by mikv_decode_attention.
 * Errors: INVALID_ARG, CAPACITY (length > max_len).
 */
int mikv_importance_update(const mikv_cache *c, int32_t length, const float *probs_hi, void *stream);

/*
 * Importance update over position-indexed rows (the same H2O accumulation,
 * Sections 3.1 and 4.1, for callers that keep scores by token position):
 *   acc[b, k, j] += ((probs[b, kG, j] + probs[b, kG+1, j]) + ...)
 * for j < length, the G = q_heads / kv_heads query heads of KV head k
 * summed left to right in fp32, then one fp32 add.
 *   acc    fp32 [batch, kv_heads, max_len] (in/out; positions >= length
 *          untouched);
 *   probs  fp32 [batch, q_heads, max_len] (e.g. mikv_probs_by_position's
 *          output when max_len = length).
 * length 0 does nothing.  Errors: INVALID_ARG (NULL pointer, a count < 1,
 * q_heads not a multiple of kv_heads, length < 0), CAPACITY (length >
 * max_len).
 */
int mikv_importance_update_positions(float *acc, const float *probs, int32_t batch, int32_t q_heads,
                                     int32_t kv_heads, int32_t length, int32_t max_len, void *stream);

/*
 * Re-rank and demote (Fig. 3 right, Section 3.1): per head, the recent
 * window is positions [length - window, length); eligible tokens are the
 * importance-pool tokens outside the window.  The k_heavy eligible tokens
 * with the largest key (score, position) stay; every other eligible token is
 * demoted: its stored high-precision key/value (fp16, or INT8/INT4 decoded
 * in fp32) is re-quantized with Eq. 1 at lo_bits into the retained pool
 * (keys are already balanced; with lo_bits 0 it is dropped instead), its
 * map entry set to 0, and its importance slot is
 * refilled from the end of the pool.  Demotion is one way.
 *   heavy_idx int32 [B, Hkv, k_heavy] or NULL (output): the positions of the
 *             kept eligible tokens (the heavy hitters), most important
 *             first by the same key (score descending, an exact score tie
 *             to the larger position); entries past the number kept are -1.
 *             Requires cap_hi <= 8192 (UNSUPPORTED otherwise).
 *   workspace at least mikv_select_workspace_size(c) bytes.
 * Errors: INVALID_ARG (k_heavy < 0, window < 0, length > max_len), CAPACITY,
 * UNSUPPORTED (heavy list with cap_hi > 8192).
 */
size_t mikv_select_workspace_size(const mikv_cache *c);
int mikv_select_topk(const mikv_cache *c, int32_t length, int32_t k_heavy, int32_t window,
                     int32_t *heavy_idx, void *workspace, size_t workspace_bytes, void *stream);

/*
 * High-precision budget of the re-rank (Section 3.1: a fixed ratio of the
 * cache kept at high precision; Fig. 3 right): the number of tokens outside
 * the recent window kept for their accumulated attention in a cache of
 * `length` tokens,
 *   k_heavy = max(0, floor(length * ratio_num / ratio_den) - (window_in_ratio ? window : 0)),
 * in 64-bit integer arithmetic.  A host function (no device work); -1 for a
 * negative length, ratio_num or window, or ratio_den < 1.
 */
int32_t mikv_heavy_budget(int32_t length, int32_t ratio_num, int32_t ratio_den, int32_t window,
                          int32_t window_in_ratio);

/*
 * First selection after prefill: every token outside the window is eligible.
 *   scores  fp32 [n_heads, length] position-indexed initial scores;
 *   hi_mask uint8 [n_heads, length] output: 1 for the window and for the
 *           k_heavy eligible tokens with the largest key (score, position).
 * Errors: INVALID_ARG.
 */
int mikv_select_prefill(const float *scores, int32_t n_heads, int32_t length, int32_t k_heavy,
                        int32_t window, uint8_t *hi_mask, void *stream);

/*
 * One whole decode step (Fig. 3, generation phase) in a single call, in the
 * order attend, accumulate, then demote:
 *   1. mikv_quantize_kv of the new token (position length - 1, importance pool);
 *   2. mikv_decode_attention over `length` tokens;
 *   3. mikv_importance_update (skipped when MIKV_ATTN_ACCUMULATE fuses it into 2);
 *   4. mikv_select_topk(k_heavy, window).
 *   q fp16 [B, Hq, 128]; k_new, v_new fp16 [B, Hkv, 128]; other arguments as
 *   in the calls above (probs_hi is required unless MIKV_ATTN_ACCUMULATE).
 * With MIKV_ATTN_ACCUMULATE, step 1 runs inside the partial phase of step 2
 * (the wave that attends over the new token's slot writes it first), and
 * with at most 512 (sequence, KV head) pairs steps 2 (finalize phase), 3
 * and 4 run as one launch, whose block that updates a head's importance
 * scores then runs that head's re-rank (two launches in all; three above
 * 512 pairs).  n_hi counts the new token from the end of the step on;
 * results are those of the four calls.
 *   workspace    at least mikv_decode_step_workspace_size(c, length) bytes
 *                (the attention's and the select's workspaces); its
 *                contents need not be initialised;
 *   phase_events NULL, or 6 hipEvent_t (entries may be NULL) recorded on
 *                `stream` before step 1 and after steps 1, 2 (partial
 *                phase), 2 (finalize phase), 3 and 4, for profiling (with
 *                the append folded the first two events both mark the start
 *                of the partial phase; with the fused launch the last three
 *                mark its end).
 * Errors: those of the four calls, checked before the first launch where the
 * host can check them.
 */
size_t mikv_decode_step_workspace_size(const mikv_cache *c, int32_t length);
int mikv_decode_step(const mikv_cache *c, int32_t length, const uint16_t *q, const uint16_t *k_new,
                     const uint16_t *v_new, const float *balance, float scale, float *out, float *probs_hi,
                     float *probs_lo, int32_t k_heavy, int32_t window, int32_t flags, void *workspace,
                     size_t workspace_bytes, void *const *phase_events, void *stream);

/*
 * mikv_decode_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops or
 * harnesses that forbid hipMalloc): the step's workspace is a device array
 * inside the library, MIKV_DECODE_STEP_NOALLOC_MAX_WORKSPACE bytes on each
 * GPU the library runs on, held until the process ends.  The call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine); the caller
 * still passes every input and output.  Arguments and results are those of
 * mikv_decode_step, on the current device (`stream` must belong to it).
 * Every call on one GPU shares that GPU's array: calls that may overlap on
 * one GPU (other streams, other threads) race and must not be issued; calls
 * on one stream are ordered and safe.  The array keeps the last call's
 * contents; nothing in it needs clearing between calls.
 * Errors: those of mikv_decode_step; CAPACITY when
 * mikv_decode_step_workspace_size(c, length) exceeds the array; HIP when the
 * array's address cannot be obtained.
 */
#define MIKV_DECODE_STEP_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)
int mikv_decode_step_noalloc(const mikv_cache *c, int32_t length, const uint16_t *q, const uint16_t *k_new,
                             const uint16_t *v_new, const float *balance, float scale, float *out, float *probs_hi,
                             float *probs_lo, int32_t k_heavy, int32_t window, int32_t flags,
                             void *const *phase_events, void *stream);

/*
 * Measurement utility (not part of the method): reads `bytes` of device
 * memory from `buf` and nothing else.  Each block of 256 threads reads one
 * contiguous chunk (at most 8192 chunks) with 16-byte loads, four in flight
 * per thread; chunks that start inside the leading `resident_bytes` are read
 * with plain loads, the others with non-temporal loads, as the attention
 * reads its resident and streamed rows (mikv_resident_bytes).  Chunks are
 * dispatched front to back, or back to front when `backwards` is non-zero
 * (alternating the two, as consecutive decode steps alternate their order).
 * Timed by the caller, it gives the read bandwidth a plain kernel reaches on
 * the device: with `resident_bytes` 0 over a buffer larger than the 256 MB
 * last-level cache, HBM's; over a decode step's bytes with the attention's
 * split, the ceiling that kernel's roofline figures are read against, next to
 * the data-sheet peak.  `buf` 16-byte aligned, `bytes` a positive multiple
 * of 16; `sink` one device uint32, written only when the XOR fold of every
 * word read equals an internal constant (it keeps the loads alive; callers
 * ignore it).
 * Errors: INVALID_ARG.
 */
int mikv_stream_read_probe(const void *buf, size_t bytes, size_t resident_bytes, int32_t backwards,
                           uint32_t *sink, void *stream);

/*
 * Bytes of a cache that the attention partial phase reads with plain loads
 * each step, importance pool first, then retained-pool heads (whole heads of
 * a pool, in head order, while they fit); every other row is read with
 * non-temporal loads.  The plain reads are what the 256 MB last-level cache
 * keeps from one decode step to the next; the non-temporal ones do not push
 * them out.  Default 224 MiB: right for one cache decoded step after step.
 * A caller that runs several caches per step (one per layer) shares the
 * last-level cache among them and should give each a part of it, or 0.
 * The setting is process-wide and takes effect at the next launch.  It
 * decides which loads are plain, and, when a cache's whole fp16 importance
 * pool lies inside it with one query head per KV head, that pool is split
 * into longer chunks (fast from the last-level cache, slower from HBM):
 * results then differ only in fp32 summation order.  Workspace sizes do not
 * depend on it.  Set it while no other thread launches decode calls, and
 * not between the _partial and _finalize calls of one attention.
 * mikv_set_resident_bytes errors: INVALID_ARG above 2^62 bytes.
 */
size_t mikv_resident_bytes(void);
int mikv_set_resident_bytes(size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* MIKV_H */
