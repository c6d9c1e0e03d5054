/*
 * spot.h -- C ABI of the SpotAttention hot path for MI355X (gfx950).
 *
 * One decode step of a full-attention layer is
 *   spot_selector_score  -> block scores of every KV block       (Section 2.1)
 *   spot_select_blocks   -> dual top-p / top-K block set          (Section 2.3)
 *   spot_sparse_decode   -> GQA attention over the chosen blocks  (Section 2)
 * with spot_decode_step running all three for every sequence in one launch,
 * spot_dense_decode as the full-attention baseline and spot_sparse_prefill
 * as the block-sparse causal prefill over query blocks.
 * spot_selector_score_tokens replaces the first call when the selector cache
 * holds one key per token (block value = maximum of per-token scores,
 * Section 2.3; spot_selector_score_tokens_blk and spot_sparse_decode_blk take
 * the paper's 16-token selector block), and spot_selector_score_q when the selector queries are
 * stored in an MX format.  Before them, spot_selector_project produces the step's
 * selector query, weights and new cache key from the hidden state, and
 * spot_selector_pool refreshes the pooled key of the block it landed in.
 *
 * Conventions shared by every entry point:
 *  - Pointers named as device arrays are caller-owned device memory; the
 *    library never allocates or frees, synchronises only in
 *    spot_decode_step_status, and between calls keeps only two process-wide
 *    values of its own: a per-device cache of the fused step's occupancy
 *    (the same number whichever call stores it) and the test hook of
 *    spot_test_force_expiry.  The decode workspaces carry completion
 *    counters and hand-off records that each call returns to zero.  Arrays
 *    are C-contiguous and start on a 16-byte boundary (as every hipMalloc and torch allocation does; the
 *    kernels read them with 16-byte vector loads).  BF16 arrays hold bfloat16
 *    values (2 bytes each).  A KV block is 64 consecutive tokens; the
 *    pooled selector key cache holds one key per block, the per-token cache
 *    one key per token.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *    enqueues work on it and returns; the returned status covers argument
 *    validation and the launch itself.  A fault inside a kernel surfaces at
 *    the caller's next synchronisation.
 *  - Arguments are validated before anything is enqueued.  On any non-zero
 *    status nothing was enqueued and no output was touched.
 *  - Calls are re-entrant; calls on different streams may run concurrently
 *    as long as they do not share output or workspace buffers.
 */
#ifndef SPOT_H
#define SPOT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t spot_status;

#define SPOT_OK 0
#define SPOT_ERR_NULL 1        /* a required pointer is NULL                      */
#define SPOT_ERR_SHAPE 2       /* a size or shape is out of range / inconsistent  */
#define SPOT_ERR_UNSUPPORTED 3 /* a valid but unimplemented size or format        */
#define SPOT_ERR_RULE 4        /* selection rule parameters are invalid           */
#define SPOT_ERR_WORKSPACE 5   /* the workspace is missing, too small or not      */
                               /* 16-byte aligned                                 */
#define SPOT_ERR_HIP 6         /* the HIP runtime reported a launch error         */
#define SPOT_ERR_EXPIRED 7     /* a bounded wait of the fused decode step expired */
                               /* (reported by spot_decode_step_status)           */

/* Storage formats of the selector key cache (Section 5.3, Appendix G: INT8,
 * FP8 and group-32 microscale 4-bit formats alongside BF16; here every
 * quantized format carries one scale per 32 elements). */
#define SPOT_KFMT_BF16 0
#define SPOT_KFMT_INT4_G32 1  /* signed 4-bit codes, FP16 scale per 32 elements */
#define SPOT_KFMT_MXFP4_G32 2 /* OCP MXFP4: E2M1 codes, E8M0 scale per 32       */
#define SPOT_KFMT_INT8_G32 3  /* signed 8-bit codes, FP16 scale per 32 elements */
#define SPOT_KFMT_MXFP8_G32 4 /* OCP MXFP8: E4M3 codes, E8M0 scale per 32       */

/* Human-readable name of a status code (static storage). */
const char *spot_status_str(spot_status s);

/* Library version string (static storage). */
const char *spot_version(void);

/*
 * spot_selector_project -- the selector's query, key and weight projections.
 *
 * Section 2.1: the selector projects the hidden state h of a token into
 * per-head query and key vectors q^I = W_q h, k^I = W_k h (h_s heads of d_s
 * dims) and per-head mixing weights w = W_w h.  Appendix A: rotary position
 * embedding covers rope_dim (64) of the head dims; here the first rope_dim
 * dims of every head, rotated in pairs (i, i + rope_dim/2) by the angle
 * pos * rope_base^(-2i / rope_dim) (the rotate-half convention), after the
 * projection and before rounding.  For each row r:
 *     q_out[r]  = RoPE(W_q h[r], pos[r])               (BF16, round to nearest even)
 *     w_out[r]  = W_w h[r]                             (FP32)
 *     k_cache[r / rows_per_seq, pos[r]] = RoPE(W_k h[r], pos[r])  (BF16), the
 *     append to the per-token selector cache; a row with pos outside
 *     [0, l_cap) stores no key.
 * Decode passes one row per sequence (rows_per_seq = 1, pos = the new
 * token's position); prefill may pass every token of a sequence
 * (rows_per_seq = L, pos = 0 .. L-1).
 *
 *  h        device BF16 [rows, d_model], 16-byte aligned, d_model % 8 == 0
 *  w_q, w_k device BF16 [h_s*d_s, d_model] (output-major, as a linear layer
 *           stores its weight), 16-byte aligned
 *  w_w      device BF16 [h_s, d_model], 16-byte aligned
 *  pos      device int32 [rows]
 *  q_out    device BF16 [rows, h_s, d_s] (output)
 *  w_out    device float [rows, h_s] (output)
 *  k_cache  device BF16 [rows/rows_per_seq, l_cap, h_s, d_s] (the rows at pos
 *           are written)
 *
 * Supported: h_s * d_s == 512 with d_s in {64, 128}; rope_dim even, 0 <=
 * rope_dim <= d_s; rope_base > 0.  The arithmetic is FP32 (products of
 * BF16, fixed summation order); the rotation angle (position times the
 * pair's frequency rope_base^(-2i/rope_dim), both in FP64) is reduced modulo
 * 2 pi in FP64, its sine and cosine taken in FP32.  Errors:
 * SPOT_ERR_NULL, SPOT_ERR_SHAPE (sizes, rows % rows_per_seq, alignment),
 * SPOT_ERR_UNSUPPORTED (head shape, rope_dim, rope_base).
 */
spot_status spot_selector_project(const void *h, const void *w_q, const void *w_k,
                                  const void *w_w, const int32_t *pos, int rows, int d_model,
                                  int h_s, int d_s, int rope_dim, float rope_base, void *q_out,
                                  float *w_out, void *k_cache, int rows_per_seq, int l_cap,
                                  void *stream);

/*
 * spot_selector_project_pooled -- one decode step's selector front end in a
 * single launch: spot_selector_project with one row per sequence
 * (rows = n_seq, rows_per_seq = 1), then spot_selector_pool of the block the
 * new key landed in (first_block = pos / 64, max_blocks = 1), with the same
 * arithmetic and summation order, so q_out, w_out, k_cache and k_pool are
 * bit for bit those of the two calls (Section 2.1: the new token's selector
 * key joins the per-token cache and the pooled key of its block is the mean
 * of the block's token keys).
 *
 *  pos      device int32 [n_seq]: the new token's position (no key stored or
 *           pooled outside [0, l_cap))
 *  seq_len  device int32 [n_seq] or NULL (pos + 1): tokens below it count in
 *           the pooled mean
 *  k_pool   device BF16 [n_seq, l_cap/64, h_s, d_s] (output), 16-byte aligned
 *  the rest as spot_selector_project.
 *
 * Errors: those of spot_selector_project; SPOT_ERR_NULL for k_pool,
 * SPOT_ERR_SHAPE when l_cap % 64 != 0.
 */
spot_status spot_selector_project_pooled(const void *h, const void *w_q, const void *w_k,
                                         const void *w_w, const int32_t *pos,
                                         const int32_t *seq_len, int n_seq, int d_model,
                                         int h_s, int d_s, int rope_dim, float rope_base,
                                         void *q_out, float *w_out, void *k_cache, void *k_pool,
                                         int l_cap, void *stream);

/*
 * spot_selector_pool -- block-pooled selector keys from the per-token cache.
 *
 * The pooled cache (one key per 64-token block, the key side of the
 * query-block x key-block tiles of Section 2.1) holds the mean of the block's
 * token keys: for each sequence b and block j = first_block[b] + y,
 * y = 0 .. max_blocks-1,
 *     k_pool[b, j] = BF16( (sum over t in block j, t < seq_len[b], of
 *                           k_tok[b, t], in FP32) / count )
 * where each 16-token quarter of the block is summed in FP32 as a pairwise
 * tree ((t0 + t1) + (t2 + t3), then groups of 4 and of 8; absent tokens count
 * as -0.0) and the four quarter sums are added in order (deterministic).
 * Blocks with no token below seq_len, or outside [0, l_cap/64), are left
 * untouched.  Decode re-pools only the block the new token fell in
 * (first_block = (seq_len - 1) / 64, max_blocks = 1); prefill pools all
 * (first_block NULL = 0, max_blocks = l_cap / 64).
 *
 *  k_tok        device BF16 [n_seq, l_cap, h_s, d_s], 16-byte aligned
 *  k_pool       device BF16 [n_seq, l_cap/64, h_s, d_s] (output), 16-byte aligned
 *  seq_len      device int32 [n_seq] or NULL (all l_cap tokens exist)
 *  first_block  device int32 [n_seq] or NULL (0)
 *
 * Supported: h_s * d_s == 512, max_blocks <= 65535.
 */
spot_status spot_selector_pool(const void *k_tok, void *k_pool, int n_seq, int l_cap, int h_s,
                               int d_s, const int32_t *seq_len, const int32_t *first_block,
                               int max_blocks, void *stream);

/*
 * spot_selector_score -- block scores of the learned selector.
 *
 * Section 2.1: the selector's score of a key for a query is the head-weighted
 * ReLU score  s = sum_h w_h * ReLU(q_h . k_h), computed once per
 * query-block x key-block tile.  Here the key side of a tile is the block's
 * pooled selector key k_bar[b, j, h, :], so
 *     scores[r, j] = sum_{h < h_s} w[r, h] * max(0, sum_{i < d_s} q_sel[r, h, i] * k_bar[seq(r), j, h, i])
 * with no 1/sqrt(d_s) factor (temperature 1).  Rows r = 0 .. n_seq*rows_per_seq-1
 * and seq(r) = r / rows_per_seq: decode uses rows_per_seq = 1 (one query per
 * sequence); prefill uses rows_per_seq = number of query blocks, with q_sel
 * and w holding query-block pooled selector queries and weights.
 *
 *  q_sel    device, BF16 [n_seq*rows_per_seq, h_s, d_s]
 *  w        device, float [n_seq*rows_per_seq, h_s]
 *  k_sel    device, selector key cache, [n_seq, nblk, h_s, d_s] BF16 for
 *           SPOT_KFMT_BF16; for the 4-bit formats uint8 [n_seq, nblk, h_s, d_s/2]
 *           with element 2i in the low nibble of byte i; for the 8-bit
 *           formats uint8 [n_seq, nblk, h_s, d_s], one code per byte
 *  k_scale  device, NULL for BF16; else [n_seq, nblk, h_s, d_s/32]: FP16 for
 *           INT4 / INT8 (value = code * scale, the code a two's-complement
 *           nibble / byte), uint8 E8M0 for MXFP4 / MXFP8 (value =
 *           E2M1(code) or E4M3(code) times 2^(e - 127))
 *  n_valid  device int32 [rows] (blocks j >= n_valid[r] do not exist and score
 *           -inf) or NULL (every block valid)
 *  scores   device, float [rows, nblk]  (output)
 *
 * Supported: h_s * d_s == 512 with d_s in {64, 128}, any format and any
 * rows_per_seq (BF16 keys with rows_per_seq a multiple of 16 run on the
 * matrix cores, everything else on the vector units).
 */
spot_status spot_selector_score(const void *q_sel, const float *w, const void *k_sel,
                                const void *k_scale, int kfmt, int n_seq, int rows_per_seq,
                                int nblk, int h_s, int d_s, const int32_t *n_valid,
                                float *scores, void *stream);

/*
 * spot_selector_score_q -- block scores with quantized selector queries.
 *
 * Section 5.3 and Appendix G quantize the selector's queries as well as its
 * key cache (INT8, INT4, FP8 and FP4).  The score is that of
 * spot_selector_score, with q_sel given as codes in the layouts of the key
 * cache formats (32-element groups along each row of h_s * d_s = 512):
 *   qfmt SPOT_KFMT_INT4_G32  : uint8 [rows, h_s, d_s/2] two's-complement
 *                              nibbles (element 2i low), q_scale FP16 bits
 *                              uint16 [rows, h_s, d_s/32];
 *   qfmt SPOT_KFMT_INT8_G32  : int8 [rows, h_s, d_s], q_scale as for INT4;
 *   qfmt SPOT_KFMT_MXFP4_G32 : E2M1 codes, uint8 [rows, h_s, d_s/2] (element
 *                              2i low), q_scale uint8 E8M0 [rows, h_s, d_s/32];
 *   qfmt SPOT_KFMT_MXFP8_G32 : E4M3 codes, uint8 [rows, h_s, d_s], q_scale as
 *                              for MXFP4;
 * an element's value is code * scale of its group.  qfmt SPOT_KFMT_BF16 is
 * spot_selector_score itself (q_scale ignored).  Keys in any format.
 *
 * When queries and keys share one MX format, d_s == 128 and rows_per_seq is
 * a multiple of 16 (prefill's query blocks), each head's tile product runs on
 * the matrix cores' block-scaled instruction (v_mfma_scale_f32_16x16x128_f8f6f4:
 * E2M1 or E4M3 operands, the E8M0 scales applied per 32-element group in
 * hardware).  Otherwise MX queries are decoded exactly in registers, and
 * integer queries enter the dot product as their integer codes, each lane's
 * partial sum (8 elements of one group) then multiplied by the group's
 * scale.  All paths accumulate in FP32.
 *
 * Errors: SPOT_ERR_NULL (a pointer, q_scale, or k_scale for quantized keys),
 * SPOT_ERR_SHAPE, SPOT_ERR_UNSUPPORTED (unknown query or key format, head
 * shape).
 */
spot_status spot_selector_score_q(const void *q_sel, const void *q_scale, int qfmt,
                                  const float *w, const void *k_sel, const void *k_scale,
                                  int kfmt, int n_seq, int rows_per_seq, int nblk, int h_s,
                                  int d_s, const int32_t *n_valid, float *scores, void *stream);

/*
 * spot_selector_score_tokens -- per-token selector, one value per block.
 *
 * Section 2.3: both selection modes rank a block by the largest per-token
 * selector score among its tokens.  With one selector key per token (the
 * score of Section 2.1 against each token's own key) and blocks of 64 tokens:
 *     scores[r, b] = max_{64b <= t < min(64b + 64, seq_len[r])}
 *                    sum_{h < h_s} w[r, h] * max(0, q_sel[r, h, :] . k_tok[seq(r), t, h, :])
 * and -inf for a block with no visible token.  Rows and seq(r) as in
 * spot_selector_score.  The result feeds spot_select_blocks unchanged
 * (n_valid[r] = ceil(seq_len[r] / 64)).
 *
 *  q_sel    device, BF16 [n_seq*rows_per_seq, h_s, d_s]
 *  w        device, float [n_seq*rows_per_seq, h_s]
 *  k_tok    device, per-token selector key cache, [n_seq, l_cap, h_s, d_s] BF16
 *           for SPOT_KFMT_BF16; the quantized formats as for
 *           spot_selector_score with one row per token instead of per block
 *           (4-bit: [n_seq, l_cap, h_s, d_s/2] uint8; 8-bit: [.., d_s] uint8)
 *  k_scale  device, NULL for BF16; else [n_seq, l_cap, h_s, d_s/32] (FP16 for
 *           INT4 / INT8, uint8 E8M0 for MXFP4 / MXFP8)
 *  l_cap    tokens per sequence in the cache, a multiple of 64; nblk = l_cap/64
 *  seq_len  device int32 [rows]: row r sees tokens t < seq_len[r] (clamped to
 *           [0, l_cap]); NULL means every token is visible
 *  scores   device, float [rows, nblk] (output)
 *
 * Supported: h_s * d_s == 512 with d_s in {64, 128}, any format.  Rows of one
 * sequence are scheduled on the same XCD so that they share its L2 for the
 * key stream.  Errors: SPOT_ERR_NULL for a missing pointer (or missing scales
 * of a 4-bit format), SPOT_ERR_SHAPE for negative sizes or l_cap not a
 * multiple of 64, SPOT_ERR_UNSUPPORTED for other head shapes or formats.
 * Nothing is written on an error.
 */
spot_status spot_selector_score_tokens(const void *q_sel, const float *w, const void *k_tok,
                                       const void *k_scale, int kfmt, int n_seq,
                                       int rows_per_seq, int l_cap, int h_s, int d_s,
                                       const int32_t *seq_len, float *scores, void *stream);

/*
 * spot_selector_score_tokens_blk -- the per-token selector with blocks of
 * blk tokens: the paper's selector block of 16 tokens (Appendix A,
 * hyper-parameter table: block size 16) or the 64-token KV block.
 *
 * Section 2.3 as for spot_selector_score_tokens, with blocks of blk tokens:
 *     scores[r, b] = max_{blk*b <= t < min(blk*b + blk, seq_len[r])} (token score of t)
 * and -inf for a block with no visible token; nblk = l_cap / blk, and
 * spot_select_blocks takes the result with n_valid[r] = ceil(seq_len[r] /
 * blk).  Arguments, layouts and errors as for spot_selector_score_tokens (l_cap
 * a multiple of 64 in both cases), plus
 *
 *  blk      16 or 64 (spot_selector_score_tokens is blk = 64); anything else
 *           is SPOT_ERR_UNSUPPORTED
 *  scores   device, float [rows, l_cap / blk] (output)
 *
 * The key stream is the same as with 64-token blocks; each 16-token block's
 * maximum is taken over the same per-token scores, so the 64-token value of
 * a block is the largest of its four 16-token values, bit for bit.
 */
spot_status spot_selector_score_tokens_blk(const void *q_sel, const float *w, const void *k_tok,
                                           const void *k_scale, int kfmt, int n_seq,
                                           int rows_per_seq, int l_cap, int blk, int h_s,
                                           int d_s, const int32_t *seq_len, float *scores,
                                           void *stream);

/*
 * spot_select_blocks -- dual top-p / static top-K block selection.
 *
 * Section 2.3 (Eqs. select-topk, select-nucleus, select-topp).  Per row r,
 * over the valid blocks [0, nv) with nv = n_valid[r] (or nblk):
 *  1. reserved R = sink prefix [0, n_sink) u recency suffix [nv-n_recent, nv);
 *  2. residual softmax p~ over B_res = [0, nv) \ R (reserved blocks excluded);
 *  3. nucleus = the smallest prefix of B_res in descending score order (equal
 *     scores: lower block id first) whose cumulative p~ reaches top_p
 *     (inclusive); top_p >= 1 takes all of B_res, top_p <= 0 none;
 *  4. cap |R| + |nucleus| <= k_max, then floor |S| >= k_min by extending the
 *     nucleus along the same order (never past k_max or |B_res|).
 * Static top-K is top_p = 1, n_sink = n_recent = 0, k_max = K.
 *
 *  scores    device float [rows, nblk] (entries j >= nv are ignored)
 *  n_valid   device int32 [rows] or NULL
 *  idx       device int32 [rows, k_max] (output): S in ascending block id,
 *            padded with -1
 *  count     device int32 [rows] (output): |S|
 *  nuc_mass  device float [rows] (output, may be NULL): p~-mass of the nucleus
 *
 * Errors: SPOT_ERR_RULE if top_p is NaN, k_max < 1, k_min > k_max,
 * n_sink < 0, n_recent < 0 or k_max < n_sink + n_recent; SPOT_ERR_UNSUPPORTED
 * if nblk > 16384 or k_max > 4096.  Deterministic: the same scores give the
 * same outputs bit for bit.
 */
spot_status spot_select_blocks(const float *scores, int rows, int nblk, const int32_t *n_valid,
                               float top_p, int k_max, int k_min, int n_sink, int n_recent,
                               int32_t *idx, int32_t *count, float *nuc_mass, void *stream);

/*
 * Workspace bytes that spot_sparse_decode (max_blocks = k_max) and
 * spot_dense_decode (max_blocks = l_cap / 64) need for these sizes: split
 * partials (float) followed by one completion counter per (sequence, KV
 * head).  Returns 0 for non-positive sizes.
 */
size_t spot_decode_workspace_bytes(int batch, int h_q, int h_kv, int d, int max_blocks);

/*
 * spot_sparse_decode -- GQA decode attention over the selected blocks only.
 *
 * Section 2 and the method figure: the layer attends only to the keys and
 * values of the selected block set S (one set per sequence, shared by every
 * head).  For sequence b and query head h with KV head g = h / (h_q / h_kv):
 *     out[b, h] = sum_{t in T} softmax_t(sm_scale * q[b,h] . k[b,g,t]) v[b,g,t],
 *     T = { t < seq_len[b] : t / 64 in S_b },  lse[b, h] = log sum_{t in T} exp(.)
 * Entries of idx that are negative or whose block starts at or past seq_len
 * are skipped, so a bad index cannot cause an out-of-bounds read.  An empty
 * T gives out = 0 and lse = -inf.  The work split and every reduction order
 * depend only on the sizes, so identical inputs give bitwise identical
 * outputs.
 *
 *  q        device BF16 [batch, h_q, d]
 *  k, v     device BF16 [batch, h_kv, l_cap, d]  (l_cap a multiple of 64)
 *  seq_len  device int32 [batch] (values above l_cap are clamped to l_cap)
 *  idx      device int32 [batch, k_max] distinct block ids, any order
 *  count    device int32 [batch] number of leading entries of idx to use
 *  out      device BF16 [batch, h_q, d] (output, round to nearest even)
 *  lse      device float [batch, h_q] (output, may be NULL)
 *  ws       device workspace of at least
 *           spot_decode_workspace_bytes(batch, h_q, h_kv, d, k_max) bytes,
 *           16-byte aligned.  It must be zero-filled before its first use;
 *           every call leaves it ready for the next one (its completion
 *           counters return to zero).  Where the counters lie depends on
 *           batch, h_q, h_kv and k_max (not on the block size of
 *           spot_sparse_decode_blk), so a workspace reused with other
 *           sizes must be zero-filled again first.  Calls that may overlap
 *           in time need separate workspaces.
 *
 * Supported: d == 128, h_q a multiple of h_kv with h_q / h_kv <= 16 (the
 * group's heads are the columns of the 16-wide matrix tiles).
 */
spot_status spot_sparse_decode(const void *q, const void *k, const void *v,
                               const int32_t *seq_len, const int32_t *idx, const int32_t *count,
                               int k_max, int batch, int h_q, int h_kv, int d, int l_cap,
                               float sm_scale, void *out, float *lse, void *ws, size_t ws_bytes,
                               void *stream);

/*
 * spot_sparse_decode_blk -- spot_sparse_decode over blocks of blk tokens:
 * the paper's 16-token selector block (Appendix A) or the 64-token KV block.
 *
 * Section 2 and the method figure, with T = { t < seq_len[b] : t / blk in
 * S_b }: the layer attends to the tokens of the selected blocks of blk
 * tokens each.  Arguments, layouts, workspace and errors as for
 * spot_sparse_decode (which is blk = 64); idx holds ids of blk-token
 * blocks, and entries that are negative or start at or past seq_len are
 * skipped.
 *
 *  blk      16 or 64; anything else is SPOT_ERR_UNSUPPORTED
 *  ws       at least spot_decode_workspace_bytes(batch, h_q, h_kv, d, k_max)
 *           bytes, as for spot_sparse_decode
 *
 * With 16-token blocks each wave of a workgroup streams one 16-row slice of
 * a block per step, the same 4 KiB contiguous K and V reads as with 64-token
 * blocks, so the HBM stream is unchanged.
 */
spot_status spot_sparse_decode_blk(const void *q, const void *k, const void *v,
                                   const int32_t *seq_len, const int32_t *idx,
                                   const int32_t *count, int k_max, int blk, int batch, int h_q,
                                   int h_kv, int d, int l_cap, float sm_scale, void *out,
                                   float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * spot_decode_step -- one decode step of the whole method for every sequence:
 * spot_selector_score (rows = batch, one query row per sequence, nblk =
 * l_cap / 64), spot_select_blocks on those scores, then spot_sparse_decode
 * on the selected blocks (Section 2: score every KV block, select by the
 * dual top-p / top-K rule with sink and recency reserved, attend to the
 * selected blocks only).  The arguments mean exactly what they mean in those
 * three calls, and the outputs (scores, idx, count, nuc_mass, out, lse) are
 * the ones they would produce.
 *
 * When h_q is 4 or 8 times h_kv, nblk <= 4096 and min(k_max, nblk) <= 512,
 * the three stages run as one launch with no kernel boundary in between: the
 * first workgroups score chunks of their sequence's blocks, one workgroup
 * per sequence selects its blocks from the scores of all chunks and
 * publishes the set, and every workgroup attends to its share of the set of
 * its (sequence, KV head) pair; the last workgroup of a pair to finish
 * merges the pair's partials.  The hand-offs go through self-flagging record words
 * in the workspace, which each reader clears again.  Otherwise (or when no
 * such grid fits) the three stages are launched one after the other on
 * `stream`.  Either way the results are deterministic; the fused path may
 * split the attention over fewer workgroups when fewer fit, which changes
 * the FP32 summation order (not the block set).
 *
 * Residency contract of the fused launch.  Its grid is sized to the number
 * of workgroups the device holds at once, and workgroups wait for records
 * written by others of the same launch: a sequence's selecting workgroup
 * waits for the scores of the sequence's scoring workgroups, and every
 * workgroup waits for its sequence's selected set.  (The merge waits for
 * nothing: the last finisher reads partials already written.)  A kernel on
 * another stream that holds compute units (or a second fused step running
 * concurrently) can keep some of these workgroups from starting.  Every wait
 * is bounded (0.2 s), so the device never hangs.  When a wait expires, the
 * waiting workgroup computes nothing on unwritten records: it attends to no
 * block, count[b] of its sequence becomes -1, and a sticky expiry word in
 * the workspace is set.  While that word is set, every later call on the
 * workspace gives count = -1 for every sequence and zero outputs (idx and
 * nuc_mass are left as they were) without waiting, until
 * spot_decode_step_status() reports the expiry and zero-fills the
 * workspace.  The word, not count, is authoritative: a sequence whose own
 * workgroups finished can still show its real count in the call that
 * expired.
 *
 *  scores   device float [batch, nblk]          (output)
 *  idx      device int32 [batch, k_max]         (output)
 *  count    device int32 [batch]                (output; -1 after an expiry)
 *  nuc_mass device float [batch] or NULL        (output)
 *  out, lse as spot_sparse_decode               (output; lse may be NULL)
 *  ws       device, spot_decode_step_workspace_bytes(batch, h_q, h_kv, d,
 *           k_max) bytes, 16-byte aligned: first a control region -- one
 *           completion counter per (sequence, KV head) pair (used by the
 *           fused launch and the separate decode alike), the expiry word
 *           (16 bytes), 4096 score record words per sequence and a 256-word
 *           bitmap per pair -- then, from a 256-byte boundary, the split
 *           partials (o [batch, h_q, n_split, 128] then (m, l)
 *           [batch, h_q, n_split, 2], FP32).  It must be zero-filled before its
 *           first use; every call leaves it ready for the next call with
 *           the same (batch, h_q, h_kv, k_max) (its counters, records and
 *           bitmaps return to zero; the partials hold data).  Zero-fill it
 *           again before using it for another such shape: the control words
 *           of one shape can lie where another left partials.  Calls that
 *           share a workspace must not overlap in time.
 */
size_t spot_decode_step_workspace_bytes(int batch, int h_q, int h_kv, int d, int k_max);

spot_status spot_decode_step(const void *q_sel, const float *w, const void *k_sel,
                             const void *k_scale, int kfmt, int h_s, int d_s,
                             const int32_t *n_valid, float top_p, int k_max, int k_min,
                             int n_sink, int n_recent, const void *q, const void *k,
                             const void *v, const int32_t *seq_len, int batch, int h_q,
                             int h_kv, int d, int l_cap, float sm_scale, float *scores,
                             int32_t *idx, int32_t *count, float *nuc_mass, void *out,
                             float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * spot_decode_step_q -- spot_decode_step with quantized selector queries
 * (Section 5.3, Appendix G: the selector's queries are quantized to the
 * precision of its key cache).  Arguments as spot_decode_step, plus q_scale
 * and qfmt: qfmt SPOT_KFMT_BF16 is spot_decode_step itself (q_scale
 * ignored); otherwise qfmt must equal kfmt and q_sel / q_scale hold the codes
 * and scales in the layout spot_selector_score_q documents (rows = batch).
 * The scores are those of spot_selector_score_q; selection and attention as
 * in spot_decode_step, fused under the same conditions.
 * Errors: those of spot_decode_step; SPOT_ERR_UNSUPPORTED when qfmt is
 * neither BF16 nor kfmt, SPOT_ERR_NULL when q_scale is NULL for codes.
 */
spot_status spot_decode_step_q(const void *q_sel, const void *q_scale, int qfmt, const float *w,
                               const void *k_sel, const void *k_scale, int kfmt, int h_s,
                               int d_s, const int32_t *n_valid, float top_p, int k_max,
                               int k_min, int n_sink, int n_recent, const void *q, const void *k,
                               const void *v, const int32_t *seq_len, int batch, int h_q,
                               int h_kv, int d, int l_cap, float sm_scale, float *scores,
                               int32_t *idx, int32_t *count, float *nuc_mass, void *out,
                               float *lse, void *ws, size_t ws_bytes, void *stream);

/*
 * spot_decode_step_static -- spot_decode_step for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, outputs and results as spot_decode_step,
 * without ws / ws_bytes: the workspace is an array of 8 MiB in the library's
 * device memory, one per GPU, held until the process ends (the first call on
 * a device looks it up and zero-fills it with a kernel on `stream`; every
 * call leaves it zeroed again).  The call allocates and frees nothing.
 * Errors: those of spot_decode_step, and SPOT_ERR_WORKSPACE when
 * spot_decode_step_workspace_bytes(batch, h_q, h_kv, d, k_max) exceeds 8 MiB.
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on the same GPU (other streams, other threads) race and give undefined
 * results.  Its expiry word is read and cleared by
 * spot_decode_step_status(NULL, ...).
 */
spot_status spot_decode_step_static(const void *q_sel, const float *w, const void *k_sel,
                                    const void *k_scale, int kfmt, int h_s, int d_s,
                                    const int32_t *n_valid, float top_p, int k_max, int k_min,
                                    int n_sink, int n_recent, const void *q, const void *k,
                                    const void *v, const int32_t *seq_len, int batch, int h_q,
                                    int h_kv, int d, int l_cap, float sm_scale, float *scores,
                                    int32_t *idx, int32_t *count, float *nuc_mass, void *out,
                                    float *lse, void *stream);

/*
 * spot_decode_step_status -- the expiry word of a fused-step workspace.
 *
 * Waits for `stream`, then reads the sticky expiry word that spot_decode_step
 * sets when one of its bounded waits expires (see the residency contract
 * above).  Returns SPOT_OK when it is clear.  When it is set, zero-fills the
 * whole workspace (spot_decode_step_workspace_bytes for these sizes) on
 * `stream`, waits for that, and returns SPOT_ERR_EXPIRED: the next
 * spot_decode_step on the workspace runs normally again.  The sizes are
 * those of the spot_decode_step calls that use ws.  ws == NULL means the
 * current device's array of spot_decode_step_static (SPOT_OK if that has not
 * been used on the device).  Errors: SPOT_ERR_SHAPE, SPOT_ERR_WORKSPACE (too
 * small or misaligned), SPOT_ERR_HIP.
 * This is the library's only synchronising call.
 */
spot_status spot_decode_step_status(void *ws, size_t ws_bytes, int batch, int h_q, int h_kv,
                                    int d, int k_max, void *stream);

/*
 * spot_test_force_expiry -- test hook, not part of the attention path.
 * While `on` is nonzero, every later fused spot_decode_step launch in this
 * process behaves as if each workgroup's wait for its sequence's scores had
 * expired at once (no waiting), so the expiry handling above can be tested
 * with every kernel exiting normally.  Process-wide; not for concurrent use.
 */
void spot_test_force_expiry(int on);

/*
 * spot_dense_decode -- the dense decode baseline.  The paper's decode
 * latency comparison (Section 3 names FlashAttention as the dense baseline;
 * Section 4.2, Table 1 times it) sets the method against dense attention
 * over every token of the cache.
 * This call is spot_sparse_decode with every block < ceil(seq_len / 64)
 * selected: for sequence b and query head h with KV head g = h / (h_q / h_kv),
 *     out[b, h] = sum_{t < seq_len[b]} softmax_t(sm_scale * q[b,h] . k[b,g,t]) v[b,g,t].
 * Same layouts, outputs, determinism and errors as spot_sparse_decode; ws of
 * spot_decode_workspace_bytes(batch, h_q, h_kv, d, l_cap / 64) bytes,
 * 16-byte aligned, zero-filled before first use (each call leaves it so).
 * l_cap == 0 is SPOT_ERR_SHAPE.
 */
spot_status spot_dense_decode(const void *q, const void *k, const void *v,
                              const int32_t *seq_len, int batch, int h_q, int h_kv, int d,
                              int l_cap, float sm_scale, void *out, float *lse, void *ws,
                              size_t ws_bytes, void *stream);

/*
 * spot_sparse_prefill -- block-sparse causal prefill.
 *
 * The paper's selector runs in the prefill regime with one selected key-block
 * set per query block (Section 2.1: one score per query-block x key-block
 * tile; Appendix B: the selector and block-sparse kernels run in prefill).
 * Query token i of query block qb (position p = 64*qb + i) attends to the
 * tokens t <= p of the key blocks selected for row (b, qb):
 *     out[b, h, p] = sum_t softmax_t(sm_scale * q[b,h,p] . k[b,g,t]) v[b,g,t]
 * with g = h / (h_q / h_kv).  Selected ids > qb contribute nothing (causal);
 * negative ids are skipped.
 *
 *  q        device BF16 [batch, h_q, L, d]
 *  k, v     device BF16 [batch, h_kv, L, d]   (L a multiple of 64)
 *  idx      device int32 [batch * L/64, k_max]: the first min(count, k_max)
 *           entries of row b*(L/64)+qb are the selected block ids, each at
 *           most once (a repeated id is attended once per occurrence); ids
 *           outside [0, qb] are skipped
 *  count    device int32 [batch * L/64] (negative counts as 0)
 *  out      device BF16 [batch, h_q, L, d] (output)
 *  lse      device float [batch, h_q, L] (output, natural log, may be NULL);
 *           a query token that sees no key gets out = 0 and lse = -inf
 *
 * Numerics: scores and the running softmax in FP32; the probabilities are
 * rounded to BF16 for the P.V product (FP32 accumulation).  No atomics: the
 * result is bitwise reproducible.
 *
 * Supported: d == 128, h_q / h_kv in {1, 2, 4, 8}, k_max <= 4096 and a
 * finite sm_scale > 0 (otherwise SPOT_ERR_UNSUPPORTED).
 */
spot_status spot_sparse_prefill(const void *q, const void *k, const void *v, int L,
                                const int32_t *idx, const int32_t *count, int k_max, int batch,
                                int h_q, int h_kv, int d, float sm_scale, void *out, float *lse,
                                void *stream);

/*
 * spot_probe_stream_read -- measurement helper, not part of the attention
 * path: reads `bytes` bytes of device memory at `buf` once with 16-byte
 * coalesced loads (the access pattern of the decode kernels) and writes one
 * checksum word per workgroup to `sink` (device, at least
 * spot_probe_sink_words() floats) so the loads cannot be elided.  Used to
 * measure the practical HBM read ceiling.  `buf` must be 16-byte aligned and
 * `bytes` a multiple of 16.
 */
spot_status spot_probe_stream_read(const void *buf, size_t bytes, float *sink, void *stream);
int spot_probe_sink_words(void);

#ifdef __cplusplus
}
#endif
#endif /* SPOT_H */
