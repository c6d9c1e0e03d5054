/*
 * spot_oracle.h -- plain FP64 CPU definition of the SpotAttention hot path.
 *
 * TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the CPU
 * baseline of the benchmark load this library.  It shares no code, header,
 * table or helper with the HIP library it checks.
 *
 * Every array is a host array in C order.  BF16 and FP16 values are passed as
 * their uint16 bit patterns and decoded exactly.  All arithmetic is double.
 */
#ifndef SPOT_ORACLE_H
#define SPOT_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Selector key-cache storage formats. */
#define ORACLE_KFMT_BF16 0
#define ORACLE_KFMT_INT4 1   /* signed 4-bit codes, FP16 scale per 32 elements */
#define ORACLE_KFMT_MXFP4 2  /* E2M1 codes, E8M0 scale per 32 elements        */
#define ORACLE_KFMT_INT8 3   /* signed 8-bit codes, FP16 scale per 32 elements */
#define ORACLE_KFMT_MXFP8 4  /* E4M3 codes, E8M0 scale per 32 elements        */

void oracle_set_threads(int n);
int oracle_get_threads(void);

/* Exact value of stored selector-key element number el (flat index). */
double oracle_key_value(const void *k_sel, const void *k_scale, int kfmt, int64_t el);

/* Block score s[r, j] = sum_h w[r,h] * max(0, q[r,h,:] . kbar[seq(r), j, h, :])
 * (Section 2.1, head-weighted ReLU score, one score per query-block x key-block
 * tile).  q_sel [rows, h_s, d_s] bf16, w [rows, h_s] f32,
 * k_sel [n_seq, nblk, h_s, d_s] (BF16) or codes [n_seq, nblk, h_s, d_s/2] with
 * scales [n_seq, nblk, h_s, d_s/32].  rows = n_seq * rows_per_seq and
 * seq(r) = r / rows_per_seq.  Entries j >= n_valid[r] are -inf.  n_valid may
 * be NULL (all nblk valid). */
void oracle_selector_score(const uint16_t *q_sel, const float *w, const void *k_sel,
                           const void *k_scale, int kfmt, int n_seq, int rows_per_seq,
                           int nblk, int h_s, int d_s, const int32_t *n_valid,
                           double *scores);

/* oracle_selector_score with the queries in a stored format as well:
 * q_sel (and q_scale) in format qfmt laid out like the keys, [rows, h_s, d_s]
 * elements (Section 5.3, Appendix G: queries and key cache quantized). */
void oracle_selector_score_qk(const void *q_sel, const void *q_scale, int qfmt, const float *w,
                              const void *k_sel, const void *k_scale, int kfmt, int n_seq,
                              int rows_per_seq, int nblk, int h_s, int d_s,
                              const int32_t *n_valid, double *scores);

/* Per-token selector scores reduced to one value per block (Section 2.3:
 * sbar[r, b] = max over the tokens t of block b of s[r, t], with s the score
 * of Section 2.1 against each token's own selector key).
 * k_tok [n_seq, l_cap, h_s, d_s] (BF16) or codes [n_seq, l_cap, h_s, d_s/2]
 * with scales [n_seq, l_cap, h_s, d_s/32]; blocks of blk tokens, nblk =
 * l_cap / blk.  Row r sees the tokens t < seq_len[r] (all l_cap if seq_len is
 * NULL); a block with none of them is -inf.  scores [rows, nblk]. */
void oracle_selector_score_tokens(const uint16_t *q_sel, const float *w, const void *k_tok,
                                  const void *k_scale, int kfmt, int n_seq, int rows_per_seq,
                                  int l_cap, int blk, int h_s, int d_s,
                                  const int32_t *seq_len, double *scores);

/* Dual top-p / top-K block selection (Section 2.3, Eqs. select-topk,
 * select-nucleus, select-topp) with a cap k_max on the total set size.
 * idx [rows, k_max] receives the chosen block ids ascending, padded with -1;
 * count [rows] their number; nuc_mass [rows] (may be NULL) the residual
 * probability mass of the chosen nucleus.  Returns 0, or -1 on bad rule. */
int oracle_select_blocks(const double *scores, int rows, int nblk, const int32_t *n_valid,
                         double top_p, int k_max, int k_min, int n_sink, int n_recent,
                         int32_t *idx, int32_t *count, double *nuc_mass);

/* Decode attention restricted to the selected blocks (Section 2, the layer
 * attends only to the keys of the selected set; Figure "method": attention
 * over the gathered K_I, V_I).  q [B, h_q, d], k/v [B, h_kv, l_cap, d] bf16,
 * seq_len [B]; idx/count as produced by oracle_select_blocks (one set per
 * sequence, shared by every head).  out [B, h_q, d], lse [B, h_q]. */
void oracle_sparse_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          const int32_t *seq_len, const int32_t *idx, const int32_t *count,
                          int k_max, int B, int h_q, int h_kv, int d, int l_cap, int blk,
                          double sm_scale, double *out, double *lse);

/* Dense decode attention over every token < seq_len (the full-attention
 * baseline).  Same layouts as oracle_sparse_decode. */
void oracle_dense_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                         const int32_t *seq_len, int B, int h_q, int h_kv, int d, int l_cap,
                         double sm_scale, double *out, double *lse);

/* Block-sparse causal prefill attention for a list of query blocks.
 * q [B, h_q, L, d], k/v [B, h_kv, L, d]; idx/count per (sequence, query
 * block) row, row = b * (L/blk) + qb.  For each (b, qb) in qrows (n_q entries,
 * each a row number), every query token i of the block attends to the tokens
 * t <= i of its selected blocks.  out [n_q, h_q, blk, d], lse [n_q, h_q, blk]. */
void oracle_sparse_prefill(const uint16_t *q, const uint16_t *k, const uint16_t *v, int L,
                           const int32_t *idx, const int32_t *count, int k_max, int B,
                           int h_q, int h_kv, int d, int blk, double sm_scale,
                           const int32_t *qrows, int n_q, double *out, double *lse);

/* Selector front end for rows of hidden states (Section 2.1: per-head query
 * and key projections q^I = W_q h, k^I = W_k h and the weight map w = W_w h;
 * Appendix A: rotary position embedding on 64 of the 128 head dims).
 * h [rows, d_model] bf16; w_q, w_k [h_s*d_s, d_model] and w_w [h_s, d_model]
 * bf16 (output-major); pos [rows].  q_out, k_out [rows, h_s, d_s] and
 * w_out [rows, h_s] in double, after the rotation of the pairs
 * (i, i + rope_dim/2), i < rope_dim/2, of every head by pos * base^(-2i/rope_dim). */
void oracle_selector_project(const uint16_t *h, const uint16_t *w_q, const uint16_t *w_k,
                             const uint16_t *w_w, const int32_t *pos, int rows, int d_model,
                             int h_s, int d_s, int rope_dim, double rope_base, double *q_out,
                             double *k_out, double *w_out);

/* Pooled selector keys: k_pool[b, j, :] = mean of k_tok[b, t, :] over the
 * tokens t of block j (blk tokens each) with t < seq_len[b] (all l_cap if
 * seq_len is NULL); 0 for a block with none.  k_tok [n_seq, l_cap, width]
 * bf16, k_pool [n_seq, l_cap/blk, width] double. */
void oracle_selector_pool(const uint16_t *k_tok, int n_seq, int l_cap, int blk, int width,
                          const int32_t *seq_len, double *k_pool);

#ifdef __cplusplus
}
#endif
#endif
