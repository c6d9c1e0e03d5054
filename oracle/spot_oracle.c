/*
 * spot_oracle.c -- plain FP64 CPU definition of the SpotAttention hot path.
 *
 * TEST INFRASTRUCTURE, not part of the product.  It is loaded only by the
 * tests, the smoke check and the CPU-baseline leg of the benchmark, and it
 * shares no code with the HIP library.  Every function is the plain
 * definition from the paper, written as loops in double precision:
 *
 *   selector score ....... Section 2.1: s = sum_h w_h ReLU(q_h . k_h), one
 *                          score per query-block x key-block tile
 *   per-token selector ... Section 2.3: the block value is the maximum of
 *                          the per-token scores of the block's tokens
 *   selector front end ... Section 2.1: per-head query / key projections of
 *                          the hidden state and the weight map W_w, with
 *                          rotary position embedding on part of each head
 *                          (Appendix A: RoPE head dim 64 of 128); block
 *                          pooling of the selector keys (mean of the block's
 *                          tokens) for the pooled cache
 *   block selection ...... Section 2.3: Eq. select-topk (static top-K),
 *                          Eq. select-nucleus (softmax over the residual
 *                          blocks), Eq. select-topp (sink + recency + nucleus,
 *                          floor K_min), plus a cap K_max on the set size
 *   sparse attention ..... Section 2 / Figure "method": attention over only
 *                          the gathered keys and values of the selected blocks
 *   dense attention ...... the full-attention baseline (Section 3)
 *
 * Stored formats are decoded exactly: BF16 and FP16 bit patterns, signed INT4
 * and INT8 codes times an FP16 group scale, and OCP MXFP4 / MXFP8 (E2M1 or
 * E4M3 codes times an E8M0 power-of-two group scale), 32 elements per group
 * (Section 5.3, Appendix G).
 *
 * Readings taken where the paper is silent (each is listed in the design
 * notes with its reason): the score has no 1/sqrt(d) factor and temperature
 * 1; blocks past n_valid do not exist; the recency blocks are the last
 * n_recent valid blocks; the residual softmax excludes the reserved blocks;
 * "reaches p" is an inclusive >=; ties in score rank the lower block id first;
 * p >= 1 keeps every residual block and p <= 0 none; k_max caps the total set
 * size (reserved blocks included) and is applied before the k_min floor.
 * Front end: the rotary part is the first rope_dim dimensions of each head,
 * rotated in pairs (i, i + rope_dim/2) by the angle pos * base^(-2i/rope_dim)
 * (the rotate-half convention of the Qwen3 backbones); w = W_w h with no
 * further scaling; a pooled key is the mean over the block's tokens that
 * exist (t < seq_len).
 */
#include "spot_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------- threads */
static int g_threads = 0;

void oracle_set_threads(int n) { g_threads = n; }

int oracle_get_threads(void) {
#ifdef _OPENMP
    return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------- stored formats */
static double bf16_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* IEEE binary16: sign, 5-bit exponent (bias 15), 10-bit fraction. */
static double f16_to_double(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 31;
    int m = h & 1023;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + m), e - 25);
    return sign ? -v : v;
}

/* OCP MX v1.0 E2M1: sign bit 3, two exponent bits (bias 1), one mantissa bit. */
static double e2m1_to_double(unsigned code) {
    int sign = (code >> 3) & 1;
    int e = (code >> 1) & 3;
    int m = code & 1;
    double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
    return sign ? -v : v;
}

/* OCP MX v1.0 E4M3: sign bit 7, four exponent bits (bias 7), three mantissa
 * bits; no infinities, S.1111.111 is NaN. */
static double e4m3_to_double(unsigned code) {
    int sign = (code >> 7) & 1;
    int e = (code >> 3) & 15;
    int m = code & 7;
    double v;
    if (e == 15 && m == 7)
        v = NAN;
    else if (e == 0)
        v = ldexp((double)m, -9);
    else
        v = ldexp(8.0 + m, e - 10);
    return sign ? -v : v;
}

/* OCP MX v1.0 E8M0: 2^(e - 127); 0xFF encodes NaN. */
static double e8m0_to_double(uint8_t e) {
    return e == 0xFF ? NAN : ldexp(1.0, (int)e - 127);
}

double oracle_key_value(const void *k_sel, const void *k_scale, int kfmt, int64_t el) {
    if (kfmt == ORACLE_KFMT_BF16)
        return bf16_to_double(((const uint16_t *)k_sel)[el]);
    if (kfmt == ORACLE_KFMT_INT8)
        return (double)((const int8_t *)k_sel)[el] *
               f16_to_double(((const uint16_t *)k_scale)[el / 32]);
    if (kfmt == ORACLE_KFMT_MXFP8)
        return e4m3_to_double(((const uint8_t *)k_sel)[el]) *
               e8m0_to_double(((const uint8_t *)k_scale)[el / 32]);
    uint8_t byte = ((const uint8_t *)k_sel)[el / 2];
    unsigned nib = (el & 1) ? (byte >> 4) : (byte & 15);
    if (kfmt == ORACLE_KFMT_INT4) {
        int code = nib >= 8 ? (int)nib - 16 : (int)nib;
        return code * f16_to_double(((const uint16_t *)k_scale)[el / 32]);
    }
    return e2m1_to_double(nib) * e8m0_to_double(((const uint8_t *)k_scale)[el / 32]);
}

/* ------------------------------------------------------- selector score */
void oracle_selector_score(const uint16_t *q_sel, const float *w, const void *k_sel,
                           const void *k_scale, int kfmt, int n_seq, int rows_per_seq,
                           int nblk, int h_s, int d_s, const int32_t *n_valid,
                           double *scores) {
    int rows = n_seq * rows_per_seq;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int r = 0; r < rows; ++r) {
        int seq = r / rows_per_seq;
        int nv = n_valid ? n_valid[r] : nblk;
        for (int j = 0; j < nblk; ++j) {
            if (j >= nv) {
                scores[(int64_t)r * nblk + j] = -INFINITY;
                continue;
            }
            double s = 0.0;
            for (int h = 0; h < h_s; ++h) {
                int64_t base = (((int64_t)seq * nblk + j) * h_s + h) * d_s;
                double dot = 0.0;
                for (int i = 0; i < d_s; ++i)
                    dot += bf16_to_double(q_sel[((int64_t)r * h_s + h) * d_s + i]) *
                           oracle_key_value(k_sel, k_scale, kfmt, base + i);
                s += (double)w[(int64_t)r * h_s + h] * (dot > 0.0 ? dot : 0.0);
            }
            scores[(int64_t)r * nblk + j] = s;
        }
    }
}

/* The same block score with the selector queries stored in a quantized
 * format too (Section 5.3 and Appendix G quantize the queries as well as the
 * key cache); qfmt/kfmt as oracle_key_value. */
void oracle_selector_score_qk(const void *q_sel, const void *q_scale, int qfmt, const float *w,
                              const void *k_sel, const void *k_scale, int kfmt, int n_seq,
                              int rows_per_seq, int nblk, int h_s, int d_s,
                              const int32_t *n_valid, double *scores) {
    int rows = n_seq * rows_per_seq;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int r = 0; r < rows; ++r) {
        int seq = r / rows_per_seq;
        int nv = n_valid ? n_valid[r] : nblk;
        for (int j = 0; j < nblk; ++j) {
            if (j >= nv) {
                scores[(int64_t)r * nblk + j] = -INFINITY;
                continue;
            }
            double s = 0.0;
            for (int h = 0; h < h_s; ++h) {
                int64_t kb = (((int64_t)seq * nblk + j) * h_s + h) * d_s;
                int64_t qb = ((int64_t)r * h_s + h) * d_s;
                double dot = 0.0;
                for (int i = 0; i < d_s; ++i)
                    dot += oracle_key_value(q_sel, q_scale, qfmt, qb + i) *
                           oracle_key_value(k_sel, k_scale, kfmt, kb + i);
                s += (double)w[(int64_t)r * h_s + h] * (dot > 0.0 ? dot : 0.0);
            }
            scores[(int64_t)r * nblk + j] = s;
        }
    }
}

/* Per-token selector with a per-block maximum (Section 2.3): each visible
 * token t gets the head-weighted ReLU score of Section 2.1 against its own
 * selector key, and a block's value is the largest score among its visible
 * tokens.  A block with no visible token does not exist (-inf). */
void oracle_selector_score_tokens(const uint16_t *q_sel, const float *w, const void *k_tok,
                                  const void *k_scale, int kfmt, int n_seq, int rows_per_seq,
                                  int l_cap, int blk, int h_s, int d_s,
                                  const int32_t *seq_len, double *scores) {
    int rows = n_seq * rows_per_seq;
    int nblk = l_cap / blk;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int r = 0; r < rows; ++r) {
        int seq = r / rows_per_seq;
        int len = seq_len ? seq_len[r] : l_cap;
        if (len > l_cap) len = l_cap;
        for (int j = 0; j < nblk; ++j) {
            double best = -INFINITY;
            for (int t = j * blk; t < (j + 1) * blk && t < len; ++t) {
                double s = 0.0;
                for (int h = 0; h < h_s; ++h) {
                    int64_t base = (((int64_t)seq * l_cap + t) * h_s + h) * d_s;
                    double dot = 0.0;
                    for (int i = 0; i < d_s; ++i)
                        dot += bf16_to_double(q_sel[((int64_t)r * h_s + h) * d_s + i]) *
                               oracle_key_value(k_tok, k_scale, kfmt, base + i);
                    s += (double)w[(int64_t)r * h_s + h] * (dot > 0.0 ? dot : 0.0);
                }
                if (s > best) best = s;
            }
            scores[(int64_t)r * nblk + j] = best;
        }
    }
}

/* ------------------------------------------------------- block selection */
typedef struct {
    double s;
    int id;
} scored_block;

/* Descending score; equal scores rank the lower block id first. */
static int by_score_desc(const void *a, const void *b) {
    const scored_block *x = (const scored_block *)a, *y = (const scored_block *)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

int oracle_select_blocks(const double *scores, int rows, int nblk, const int32_t *n_valid,
                         double top_p, int k_max, int k_min, int n_sink, int n_recent,
                         int32_t *idx, int32_t *count, double *nuc_mass) {
    if (isnan(top_p) || k_max < 1 || k_min > k_max || n_sink < 0 || n_recent < 0 ||
        k_max < n_sink + n_recent)
        return -1;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int r = 0; r < rows; ++r) {
        const double *s = scores + (int64_t)r * nblk;
        int nv = n_valid ? n_valid[r] : nblk;
        if (nv > nblk) nv = nblk;
        if (nv < 0) nv = 0;
        char *chosen = (char *)calloc((size_t)nblk + 1, 1);
        scored_block *res = (scored_block *)malloc(sizeof(scored_block) * ((size_t)nblk + 1));

        /* Reserved tier: a fixed sink prefix and a fixed recency suffix. */
        int n_reserved = 0;
        for (int j = 0; j < nv; ++j) {
            if (j < n_sink || j >= nv - n_recent) {
                chosen[j] = 1;
                ++n_reserved;
            }
        }
        /* Residual blocks B_res = B \ (S_sink u S_rec), sorted by score. */
        int n_res = 0;
        for (int j = 0; j < nv; ++j)
            if (!chosen[j]) {
                res[n_res].s = s[j];
                res[n_res].id = j;
                ++n_res;
            }
        qsort(res, (size_t)n_res, sizeof(scored_block), by_score_desc);

        double mass = 0.0;
        int n = 0;
        if (n_res > 0) {
            /* Residual softmax (Eq. select-nucleus). */
            double m = res[0].s, Z = 0.0;
            double *prob = (double *)malloc(sizeof(double) * (size_t)n_res);
            for (int i = 0; i < n_res; ++i) {
                prob[i] = exp(res[i].s - m);
                Z += prob[i];
            }
            for (int i = 0; i < n_res; ++i) prob[i] /= Z;
            /* Nucleus: the smallest prefix whose cumulative mass reaches p. */
            if (top_p >= 1.0) {
                n = n_res;
            } else if (top_p <= 0.0) {
                n = 0;
            } else {
                double cum = 0.0;
                n = n_res;
                for (int i = 0; i < n_res; ++i) {
                    cum += prob[i];
                    if (cum >= top_p) {
                        n = i + 1;
                        break;
                    }
                }
            }
            /* Total budget cap, then the K_min floor along descending score. */
            int cap = k_max - n_reserved;
            if (n > cap) n = cap;
            if (n_reserved + n < k_min) {
                int want = k_min - n_reserved;
                if (want > cap) want = cap;
                if (want > n_res) want = n_res;
                n = want;
            }
            for (int i = 0; i < n; ++i) {
                chosen[res[i].id] = 1;
                mass += prob[i];
            }
            free(prob);
        }
        int c = 0;
        for (int j = 0; j < nv; ++j)
            if (chosen[j]) idx[(int64_t)r * k_max + c++] = j;
        count[r] = c;
        for (int i = c; i < k_max; ++i) idx[(int64_t)r * k_max + i] = -1;
        if (nuc_mass) nuc_mass[r] = mass;
        free(res);
        free(chosen);
    }
    return 0;
}

/* ------------------------------------------------------------ attention */
/* Softmax attention of one query row over a token list; the plain
 * definition o = sum_t softmax_t(scale * q.k_t) v_t, lse = log sum_t exp(.). */
static void attend(const uint16_t *qrow, const uint16_t *kbase, const uint16_t *vbase, int d,
                   const int *tok, int n_tok, double sm_scale, double *logit, double *o,
                   double *lse) {
    for (int i = 0; i < d; ++i) o[i] = 0.0;
    if (n_tok == 0) {
        *lse = -INFINITY;
        return;
    }
    double m = -INFINITY;
    for (int u = 0; u < n_tok; ++u) {
        const uint16_t *kr = kbase + (int64_t)tok[u] * d;
        double dot = 0.0;
        for (int i = 0; i < d; ++i) dot += bf16_to_double(qrow[i]) * bf16_to_double(kr[i]);
        logit[u] = sm_scale * dot;
        if (logit[u] > m) m = logit[u];
    }
    double Z = 0.0;
    for (int u = 0; u < n_tok; ++u) {
        double p = exp(logit[u] - m);
        Z += p;
        const uint16_t *vr = vbase + (int64_t)tok[u] * d;
        for (int i = 0; i < d; ++i) o[i] += p * bf16_to_double(vr[i]);
    }
    for (int i = 0; i < d; ++i) o[i] /= Z;
    *lse = m + log(Z);
}

void oracle_sparse_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                          const int32_t *seq_len, const int32_t *idx, const int32_t *count,
                          int k_max, int B, int h_q, int h_kv, int d, int l_cap, int blk,
                          double sm_scale, double *out, double *lse) {
    int group = h_q / h_kv;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int bh = 0; bh < B * h_q; ++bh) {
        int b = bh / h_q, hq = bh % h_q, g = hq / group;
        int sl = seq_len[b] < l_cap ? seq_len[b] : l_cap;
        int nb = (l_cap + blk - 1) / blk;
        /* The selected set S (one per sequence, shared by all heads). */
        char *in_set = (char *)calloc((size_t)nb + 1, 1);
        for (int i = 0; i < count[b] && i < k_max; ++i) {
            int j = idx[(int64_t)b * k_max + i];
            if (j >= 0 && j < nb) in_set[j] = 1;
        }
        int *tok = (int *)malloc(sizeof(int) * ((size_t)l_cap + 1));
        double *logit = (double *)malloc(sizeof(double) * ((size_t)l_cap + 1));
        int n_tok = 0;
        for (int t = 0; t < sl; ++t)
            if (in_set[t / blk]) tok[n_tok++] = t;
        const uint16_t *kb = k + ((int64_t)b * h_kv + g) * l_cap * d;
        const uint16_t *vb = v + ((int64_t)b * h_kv + g) * l_cap * d;
        attend(q + ((int64_t)b * h_q + hq) * d, kb, vb, d, tok, n_tok, sm_scale, logit,
               out + ((int64_t)b * h_q + hq) * d, lse + (int64_t)b * h_q + hq);
        free(logit);
        free(tok);
        free(in_set);
    }
}

void oracle_dense_decode(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                         const int32_t *seq_len, int B, int h_q, int h_kv, int d, int l_cap,
                         double sm_scale, double *out, double *lse) {
    int group = h_q / h_kv;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int bh = 0; bh < B * h_q; ++bh) {
        int b = bh / h_q, hq = bh % h_q, g = hq / group;
        int sl = seq_len[b] < l_cap ? seq_len[b] : l_cap;
        int *tok = (int *)malloc(sizeof(int) * ((size_t)l_cap + 1));
        double *logit = (double *)malloc(sizeof(double) * ((size_t)l_cap + 1));
        for (int t = 0; t < sl; ++t) tok[t] = t;
        const uint16_t *kb = k + ((int64_t)b * h_kv + g) * l_cap * d;
        const uint16_t *vb = v + ((int64_t)b * h_kv + g) * l_cap * d;
        attend(q + ((int64_t)b * h_q + hq) * d, kb, vb, d, tok, sl, sm_scale, logit,
               out + ((int64_t)b * h_q + hq) * d, lse + (int64_t)b * h_q + hq);
        free(logit);
        free(tok);
    }
}

void oracle_sparse_prefill(const uint16_t *q, const uint16_t *k, const uint16_t *v, int L,
                           const int32_t *idx, const int32_t *count, int k_max, int B,
                           int h_q, int h_kv, int d, int blk, double sm_scale,
                           const int32_t *qrows, int n_q, double *out, double *lse) {
    (void)B;
    int group = h_q / h_kv;
    int nqb = L / blk;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int task = 0; task < n_q * h_q; ++task) {
        int qi = task / h_q, hq = task % h_q, g = hq / group;
        int row = qrows[qi];
        int b = row / nqb, qb = row % nqb;
        char *in_set = (char *)calloc((size_t)nqb + 1, 1);
        for (int i = 0; i < count[row] && i < k_max; ++i) {
            int j = idx[(int64_t)row * k_max + i];
            if (j >= 0 && j < nqb) in_set[j] = 1;
        }
        int *tok = (int *)malloc(sizeof(int) * ((size_t)L + 1));
        double *logit = (double *)malloc(sizeof(double) * ((size_t)L + 1));
        const uint16_t *kb = k + ((int64_t)b * h_kv + g) * L * d;
        const uint16_t *vb = v + ((int64_t)b * h_kv + g) * L * d;
        for (int i = 0; i < blk; ++i) {
            int pos = qb * blk + i;
            /* Causal: a query token sees selected tokens at or before it. */
            int n_tok = 0;
            for (int t = 0; t <= pos; ++t)
                if (in_set[t / blk]) tok[n_tok++] = t;
            int64_t o = (((int64_t)qi * h_q + hq) * blk + i);
            attend(q + (((int64_t)b * h_q + hq) * L + pos) * d, kb, vb, d, tok, n_tok, sm_scale,
                   logit, out + o * d, lse + o);
        }
        free(logit);
        free(tok);
        free(in_set);
    }
}

/* ------------------------------------------------------------ front end */
void oracle_selector_project(const uint16_t *h, const uint16_t *w_q, const uint16_t *w_k,
                             const uint16_t *w_w, const int32_t *pos, int rows, int d_model,
                             int h_s, int d_s, int rope_dim, double rope_base, double *q_out,
                             double *k_out, double *w_out) {
    int n_out = h_s * d_s;
    int half = rope_dim / 2;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int r = 0; r < rows; ++r) {
        const uint16_t *hr = h + (int64_t)r * d_model;
        double *qr = q_out + (int64_t)r * n_out, *kr = k_out + (int64_t)r * n_out;
        /* the linear maps: out[j] = sum_i W[j, i] h[i] */
        for (int j = 0; j < n_out; ++j) {
            double aq = 0.0, ak = 0.0;
            for (int i = 0; i < d_model; ++i) {
                double x = bf16_to_double(hr[i]);
                aq += bf16_to_double(w_q[(int64_t)j * d_model + i]) * x;
                ak += bf16_to_double(w_k[(int64_t)j * d_model + i]) * x;
            }
            qr[j] = aq;
            kr[j] = ak;
        }
        for (int hh = 0; hh < h_s; ++hh) {
            double a = 0.0;
            for (int i = 0; i < d_model; ++i)
                a += bf16_to_double(w_w[(int64_t)hh * d_model + i]) * bf16_to_double(hr[i]);
            w_out[(int64_t)r * h_s + hh] = a;
        }
        /* rotary position embedding on the first rope_dim dims of each head */
        for (int hh = 0; hh < h_s; ++hh) {
            for (int i = 0; i < half; ++i) {
                double ang = (double)pos[r] * pow(rope_base, -2.0 * i / rope_dim);
                double c = cos(ang), sn = sin(ang);
                double *v[2] = {qr + hh * d_s, kr + hh * d_s};
                for (int m = 0; m < 2; ++m) {
                    double x1 = v[m][i], x2 = v[m][i + half];
                    v[m][i] = x1 * c - x2 * sn;
                    v[m][i + half] = x2 * c + x1 * sn;
                }
            }
        }
    }
}

void oracle_selector_pool(const uint16_t *k_tok, int n_seq, int l_cap, int blk, int width,
                          const int32_t *seq_len, double *k_pool) {
    int nblk = l_cap / blk;
#pragma omp parallel for schedule(dynamic) num_threads(oracle_get_threads())
    for (int task = 0; task < n_seq * nblk; ++task) {
        int b = task / nblk, j = task % nblk;
        int len = seq_len ? seq_len[b] : l_cap;
        if (len > l_cap) len = l_cap;
        int lo = j * blk, hi = (j + 1) * blk < len ? (j + 1) * blk : len;
        double *o = k_pool + (int64_t)task * width;
        for (int e = 0; e < width; ++e) {
            if (hi <= lo) {
                o[e] = 0.0;
                continue;
            }
            double acc = 0.0;
            for (int t = lo; t < hi; ++t)
                acc += bf16_to_double(k_tok[((int64_t)b * l_cap + t) * width + e]);
            o[e] = acc / (hi - lo);
        }
    }
}
