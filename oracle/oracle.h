/*
 * oracle.h -- plain fp64 CPU oracle of the verify hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * CPU-baseline leg of bench.py may load or call it.  It shares no code with
 * the HIP library: it restates the input formats from the library's public
 * contract and computes the plain definitions, slowly and obviously.
 *
 * Return value of every function: 0 on success, -1 if an argument or the
 * metadata breaks the stated input format (nothing useful is written then).
 */
#ifndef DSV_ORACLE_H
#define DSV_ORACLE_H

#include <stdint.h>

/* Attention (Sec. III-D Eq. (16) with Eqs. (10)-(11) packing).  `out` is
 * double [cap][hq][d]; every element is written (tail rows get 0). */
int oracle_verify_attn(const uint16_t *q, const int32_t *cu_qlens,
                       const uint16_t *kv_pages, const int32_t *page_table,
                       const int32_t *ctx_lens, double *out, int32_t num_reqs,
                       int32_t cap, int32_t hq, int32_t hkv, int32_t d,
                       int32_t page_size, int32_t max_pages,
                       int32_t num_pages, double scale);

/* Per-row argmax with lowest-index tie-break.  dtype 0 = fp32, 1 = bf16. */
int oracle_row_argmax(const void *logits, int32_t dtype, int32_t rows,
                      int32_t vocab, int32_t *idx_out);

/* Greedy acceptance (Sec. III-D "Prefix verifier", temperature 0). */
int oracle_accept(const void *logits, int32_t dtype, const int32_t *cu_qlens,
                  const int32_t *draft_tokens, int32_t *accept_len,
                  int32_t *next_token, int32_t num_reqs, int32_t cap,
                  int32_t vocab);

/* Stochastic prefix verifier (Sec. III-D "Prefix verifier", temperature
 * T > 0): P = softmax(logits / T) per row; candidate x_j = draft[o+j+1] is
 * accepted iff uniforms[o+j][0] < P_{o+j}(x_j); the successor is drawn by
 * inverting the cumulative distribution (index order) of P_{o+a}, without
 * the rejected candidate if there is one, at uniforms[o+a][1].  uniforms is
 * float [cap][2].  margin_accept / margin_sample (nullable) receive per
 * request the smallest distance between a uniform and the threshold it was
 * compared with, for the accept tests and for the successor draw. */
int oracle_accept_stochastic(const void *logits, int32_t dtype,
                             const int32_t *cu_qlens, const int32_t *draft_tokens,
                             const float *uniforms, double temperature,
                             int32_t *accept_len, int32_t *next_token,
                             double *margin_accept, double *margin_sample,
                             int32_t num_reqs, int32_t cap, int32_t vocab);

/* The interval [lo, hi) of cumulative probability (vocabulary order) that
 * token `token` occupies in the successor distribution of packed row `row`:
 * P = softmax(logits[row] / T), without token `removed` (-1: none),
 * renormalised. */
int oracle_successor_interval(const void *logits, int32_t dtype, int32_t row,
                              int32_t vocab, int32_t removed, double temperature,
                              int32_t token, double *lo, double *hi);

/* Acceptance predictor forward (Sec. III-C, Eq. (5)): per live row,
 * h = relu(features . W1 + b1), out = h . W2 + b2, in double precision.
 * features float [n_rows][in_dim]; W1 [in_dim][hidden]; W2 [hidden][out_dim];
 * out double [n_rows][out_dim], zero past n_live. */
int oracle_predictor_forward(const float *features, int32_t n_live, int32_t n_rows,
                             const float *w1, const float *b1, const float *w2,
                             const float *b2, int32_t in_dim, int32_t hidden,
                             int32_t out_dim, double *out);

/* ---- DVL budget allocation and flat-buffer packing (Sec. III-C) ----
 *
 * Decisions are taken in single precision, as the library takes them: each
 * prefix score is the binary32 rounding of the sigmoid evaluated in double,
 * the cumulative minimum and all comparisons act on those binary32 values,
 * and the length estimate is a binary32 sum in position order. */

/* Prefix scores and initial lengths (Alg. 1 score and seed steps, Eqs. (6)
 * and (7)).  pred_logits float [n][w-1]; writes q float [n][w] (q[i][0] = 1),
 * ell float [n] (the estimate) and k0 [n].  2 <= w <= 64. */
int oracle_dvl_scores(const float *pred_logits, int32_t n, int32_t w,
                      float *q, float *ell, int32_t *k0);

/* Budget adjustment (Eqs. (8) and (9), Alg. 1 grow and shrink loops): one
 * request at a time, lowest request index on ties.  Requires 1 <= k0 <= w and
 * n <= budget <= n*w.  Writes k [n] and the number of single-slot updates. */
int oracle_dvl_adjust(const float *q, const int32_t *k0, int32_t n, int32_t w,
                      int32_t budget, int32_t *k, int32_t *updates);

/* Offsets, packing, sentinels and tail placeholders (Eqs. (10) and (11), Alg.
 * 1 pack and sentinel steps).  k_live [n] (each in [1, w]); fields int32
 * [n_bs][w]; writes k_out [n_bs], offsets [n_bs+1] and the three packed
 * fields [m_bs].  Requires 0 <= n <= n_bs and sum(k_live) <= m_bs. */
int oracle_dvl_pack(const int32_t *k_live, int32_t n, int32_t n_bs, int32_t w,
                    int32_t m_bs, const int32_t *tokens,
                    const int32_t *positions, const int32_t *kv_refs,
                    int32_t *k_out, int32_t *offsets, int32_t *packed_tokens,
                    int32_t *packed_positions, int32_t *packed_kv_refs);

#endif
