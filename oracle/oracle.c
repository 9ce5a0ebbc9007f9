/*
 * oracle.c -- plain fp64 CPU oracle of the verify hot path of block-diffusion
 * speculative decoding (DScale).
 *
 * TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__.smoke() and the
 * CPU-baseline leg of bench.py load it.  It shares no code, header or table
 * with the HIP library.  Every floating-point step of attention and
 * acceptance is in double precision (bf16 and fp32 inputs widen to double
 * exactly); the DVL allocator takes its decisions on binary32 scores, in the
 * precision the library decides in (oracle.h).
 *
 * What is computed (the method reaches these exactly, so the oracle is the
 * plain definition written out):
 *
 *  - Verify attention.  Sec. III-D, Eq. (16): a row (i, j) is valid iff
 *    request i is live and j < k_i; a valid row reads packed row
 *    offset_i + j (Eq. (10) offsets = exclusive prefix sum of the lengths,
 *    Eq. (11) packing) and attends with request-local causal masking over
 *    the request's committed context (the historyKV gather of Alg. 2) and
 *    over its own block.  Row j of request i therefore sees logical keys
 *    t = 0 .. ctx_i + j.  Softmax is evaluated in two passes (max, then
 *    normalised weights).  GQA: query head h reads KV head h / G.
 *
 *  - Greedy acceptance.  Sec. III-D "Prefix verifier": a candidate x is
 *    accepted with probability P(x); at temperature 0 the target policy P is
 *    one-hot at its argmax, so a candidate is accepted iff it equals the
 *    target's argmax at the previous row, the first mismatch stops the
 *    prefix, and row offset_i + a_i supplies the successor.  Sec. I: the
 *    accepted tokens are the contiguous candidate prefix, anchor excluded.
 *
 *  - DVL budget allocation and flat-buffer packing.  Sec. III-C, Alg. 1 and
 *    Eqs. (6)-(11): taken step by step in the paper's order (an iteration,
 *    not a closed form); see the section at the end of this file.
 *
 * Input formats restated from the library's public contract: bf16 values
 * are the upper 16 bits of an IEEE binary32; a KV page holds, per KV head,
 * a K tile with element (slot s, dim c) at ((c/8)*16 + s)*8 + c%8 and a V
 * tile with element (s, c) at c*16 + s.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static double widen_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* K or V element of logical key t of request i (layout comment above). */
static double kv_elem(const uint16_t *kv_pages, const int32_t *page_table,
                      int32_t i, int32_t t, int32_t which, int32_t g,
                      int32_t c, int32_t hkv, int32_t d, int32_t page_size,
                      int32_t max_pages) {
  int32_t page = page_table[(int64_t)i * max_pages + t / page_size];
  int32_t s = t % page_size;
  int64_t tile = (((int64_t)page * 2 + which) * hkv + g) * (int64_t)page_size * d;
  int64_t off;
  if (which == 0)
    off = ((int64_t)(c / 8) * page_size + s) * 8 + c % 8;
  else
    off = (int64_t)c * page_size + s;
  return widen_bf16(kv_pages[tile + off]);
}

int oracle_verify_attn(const uint16_t *q, const int32_t *cu_qlens,
                       const uint16_t *kv_pages, const int32_t *page_table,
                       const int32_t *ctx_lens, double *out, int32_t num_reqs,
                       int32_t cap, int32_t hq, int32_t hkv, int32_t d,
                       int32_t page_size, int32_t max_pages,
                       int32_t num_pages, double scale) {
  if (!q || !cu_qlens || !kv_pages || !page_table || !ctx_lens || !out)
    return -1;
  if (num_reqs < 1 || cap < 1 || hq < 1 || hkv < 1 || hq % hkv != 0 ||
      d < 8 || d % 8 != 0 || page_size < 1 || max_pages < 1 || num_pages < 1)
    return -1;
  /* Input-format checks: offsets non-decreasing from 0 within capacity,
   * every page that will be read exists. */
  if (cu_qlens[0] != 0 || cu_qlens[num_reqs] > cap) return -1;
  for (int32_t i = 0; i < num_reqs; ++i) {
    int32_t k = cu_qlens[i + 1] - cu_qlens[i];
    if (k < 0 || ctx_lens[i] < 0) return -1;
    int64_t keys = (int64_t)ctx_lens[i] + k;
    if (k > 0) {
      int64_t pages = (keys + page_size - 1) / page_size;
      if (pages > max_pages) return -1;
      for (int64_t p = 0; p < pages; ++p) {
        int32_t id = page_table[(int64_t)i * max_pages + p];
        if (id < 0 || id >= num_pages) return -1;
      }
    }
  }

  const int32_t group = hq / hkv;
  memset(out, 0, sizeof(double) * (size_t)cap * hq * d);

  int32_t max_keys = max_pages * page_size;
  double *score = (double *)malloc(sizeof(double) * (size_t)max_keys);
  double *acc = (double *)malloc(sizeof(double) * (size_t)d);
  if (!score || !acc) {
    free(score);
    free(acc);
    return -1;
  }

  for (int32_t i = 0; i < num_reqs; ++i) {
    int32_t row0 = cu_qlens[i];
    int32_t k = cu_qlens[i + 1] - row0;
    for (int32_t j = 0; j < k; ++j) {
      int32_t visible = ctx_lens[i] + j + 1; /* keys 0 .. ctx_i + j */
      for (int32_t h = 0; h < hq; ++h) {
        int32_t g = h / group;
        const uint16_t *qrow = q + ((int64_t)(row0 + j) * hq + h) * d;
        /* pass 1: scores and their maximum */
        double m = -INFINITY;
        for (int32_t t = 0; t < visible; ++t) {
          double dot = 0.0;
          for (int32_t c = 0; c < d; ++c)
            dot += widen_bf16(qrow[c]) *
                   kv_elem(kv_pages, page_table, i, t, 0, g, c, hkv, d,
                           page_size, max_pages);
          score[t] = scale * dot;
          if (score[t] > m) m = score[t];
        }
        /* pass 2: weights exp(s - m), weighted sum of V, normalisation */
        double denom = 0.0;
        for (int32_t c = 0; c < d; ++c) acc[c] = 0.0;
        for (int32_t t = 0; t < visible; ++t) {
          double w = exp(score[t] - m);
          denom += w;
          for (int32_t c = 0; c < d; ++c)
            acc[c] += w * kv_elem(kv_pages, page_table, i, t, 1, g, c, hkv, d,
                                  page_size, max_pages);
        }
        double *orow = out + ((int64_t)(row0 + j) * hq + h) * d;
        for (int32_t c = 0; c < d; ++c) orow[c] = acc[c] / denom;
      }
    }
  }
  free(score);
  free(acc);
  return 0;
}

static double logit_at(const void *logits, int32_t dtype, int64_t idx) {
  if (dtype == 0) return (double)((const float *)logits)[idx];
  return widen_bf16(((const uint16_t *)logits)[idx]);
}

int oracle_row_argmax(const void *logits, int32_t dtype, int32_t rows,
                      int32_t vocab, int32_t *idx_out) {
  if (!logits || !idx_out || rows < 0 || vocab < 1 || (dtype != 0 && dtype != 1))
    return -1;
  for (int32_t r = 0; r < rows; ++r) {
    int64_t base = (int64_t)r * vocab;
    int32_t best = 0;
    double best_val = logit_at(logits, dtype, base);
    for (int32_t v = 1; v < vocab; ++v) {
      double x = logit_at(logits, dtype, base + v);
      if (x > best_val) { /* strict: the first (lowest) index keeps ties */
        best_val = x;
        best = v;
      }
    }
    idx_out[r] = best;
  }
  return 0;
}

int oracle_accept(const void *logits, int32_t dtype, const int32_t *cu_qlens,
                  const int32_t *draft_tokens, int32_t *accept_len,
                  int32_t *next_token, int32_t num_reqs, int32_t cap,
                  int32_t vocab) {
  if (!logits || !cu_qlens || !draft_tokens || !accept_len || !next_token)
    return -1;
  if (num_reqs < 1 || cap < 1 || vocab < 1) return -1;
  if (cu_qlens[0] != 0 || cu_qlens[num_reqs] > cap) return -1;
  for (int32_t i = 0; i < num_reqs; ++i)
    if (cu_qlens[i + 1] < cu_qlens[i]) return -1;

  int32_t live = cu_qlens[num_reqs];
  int32_t *target = (int32_t *)malloc(sizeof(int32_t) * (size_t)(live > 0 ? live : 1));
  if (!target) return -1;
  if (oracle_row_argmax(logits, dtype, live, vocab, target) != 0) {
    free(target);
    return -1;
  }
  for (int32_t i = 0; i < num_reqs; ++i) {
    int32_t o = cu_qlens[i];
    int32_t k = cu_qlens[i + 1] - o;
    if (k == 0) { /* sentinel request: no rows, no successor */
      accept_len[i] = 0;
      next_token[i] = -1;
      continue;
    }
    /* candidate j+1 (row o+j+1 of the inputs) survives iff the target's
     * choice at row o+j reproduces it; the first mismatch ends the prefix */
    int32_t a = 0;
    while (a < k - 1 && target[o + a] == draft_tokens[o + a + 1]) ++a;
    accept_len[i] = a;
    next_token[i] = target[o + a];
  }
  free(target);
  return 0;
}

/* ------------------------------------------------------------------------
 * DVL budget allocation and flat-buffer packing (Sec. III-C).
 *
 * Alg. 1 in the paper's order: sigmoid scores with the anchor's score fixed at
 * one and a running minimum so that scores never increase along the block
 * (Eq. (6)); the estimate is the sum of the W-1 draft scores, rounded half up
 * and clipped to [1, W] (Eq. (7)); the gap to the budget is closed one slot
 * at a time, growing the request whose next slot scores highest or shrinking
 * the one whose last slot scores lowest (Eq. (9)); offsets are the exclusive
 * prefix sum (Eq. (10)) and every field is copied to offset_i + j (Eq. (11));
 * requests past the live count get length 0 and offset M_live, and slots past
 * M_live get token 0, position 0 and the first request's first cache
 * reference.
 *
 * Readings: the paper leaves the tie-break of Eq. (9) open; here the lowest
 * request index wins.  It fixes no precision; decisions are taken on binary32
 * scores (see oracle.h).  A NaN score leaves the running minimum unchanged.
 * ---------------------------------------------------------------------- */

int oracle_dvl_scores(const float *pred_logits, int32_t n, int32_t w,
                      float *q, float *ell, int32_t *k0) {
  if (n < 0 || w < 2 || w > 64 || (n > 0 && (!pred_logits || !q || !ell || !k0)))
    return -1;
  for (int32_t i = 0; i < n; ++i) {
    float *qi = q + (int64_t)i * w;
    qi[0] = 1.0f;
    for (int32_t j = 1; j < w; ++j) {
      double x = (double)pred_logits[(int64_t)i * (w - 1) + (j - 1)];
      float sig = (float)(1.0 / (1.0 + exp(-x)));
      qi[j] = (sig < qi[j - 1]) ? sig : qi[j - 1];
    }
    float sum = 0.0f;
    for (int32_t j = 1; j < w; ++j) sum += qi[j];
    ell[i] = sum;
    float r = floorf(sum + 0.5f);
    int32_t k = r < 1.0f ? 1 : (r > (float)w ? w : (int32_t)r);
    k0[i] = k;
  }
  return 0;
}

int oracle_dvl_adjust(const float *q, const int32_t *k0, int32_t n, int32_t w,
                      int32_t budget, int32_t *k, int32_t *updates) {
  if (n < 1 || w < 2 || !q || !k0 || !k || !updates) return -1;
  if (budget < n || (int64_t)budget > (int64_t)n * w) return -1;
  int64_t sum = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (k0[i] < 1 || k0[i] > w) return -1;
    k[i] = k0[i];
    sum += k0[i];
  }
  int64_t gap = (int64_t)budget - sum;
  int32_t count = 0;
  while (gap > 0) {
    int32_t best = -1;
    for (int32_t i = 0; i < n; ++i) {
      if (k[i] >= w) continue;
      if (best < 0 || q[(int64_t)i * w + k[i]] > q[(int64_t)best * w + k[best]]) best = i;
    }
    if (best < 0) return -1; /* unreachable for a budget within [n, n*w] */
    k[best] += 1;
    gap -= 1;
    ++count;
  }
  while (gap < 0) {
    int32_t best = -1;
    for (int32_t i = 0; i < n; ++i) {
      if (k[i] <= 1) continue;
      if (best < 0 || q[(int64_t)i * w + k[i] - 1] < q[(int64_t)best * w + k[best] - 1])
        best = i;
    }
    if (best < 0) return -1;
    k[best] -= 1;
    gap += 1;
    ++count;
  }
  *updates = count;
  return 0;
}

int oracle_dvl_pack(const int32_t *k_live, int32_t n, int32_t n_bs, int32_t w,
                    int32_t m_bs, const int32_t *tokens,
                    const int32_t *positions, const int32_t *kv_refs,
                    int32_t *k_out, int32_t *offsets, int32_t *packed_tokens,
                    int32_t *packed_positions, int32_t *packed_kv_refs) {
  if (n < 0 || n_bs < 1 || n > n_bs || w < 1 || m_bs < 0) return -1;
  if (!tokens || !positions || !kv_refs || !k_out || !offsets) return -1;
  if (m_bs > 0 && (!packed_tokens || !packed_positions || !packed_kv_refs)) return -1;
  int64_t live = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (k_live[i] < 1 || k_live[i] > w) return -1;
    live += k_live[i];
  }
  if (live > m_bs) return -1;
  /* offsets of live requests, then sentinels: length 0 at offset M_live */
  offsets[0] = 0;
  for (int32_t i = 0; i < n_bs; ++i) {
    k_out[i] = i < n ? k_live[i] : 0;
    offsets[i + 1] = offsets[i] + k_out[i];
  }
  /* every live slot: the field value of (request, position) it maps to */
  for (int32_t i = 0; i < n; ++i) {
    for (int32_t j = 0; j < k_out[i]; ++j) {
      int32_t s = offsets[i] + j;
      packed_tokens[s] = tokens[(int64_t)i * w + j];
      packed_positions[s] = positions[(int64_t)i * w + j];
      packed_kv_refs[s] = kv_refs[(int64_t)i * w + j];
    }
  }
  /* tail placeholders */
  for (int64_t s = live; s < m_bs; ++s) {
    packed_tokens[s] = 0;
    packed_positions[s] = 0;
    packed_kv_refs[s] = kv_refs[0];
  }
  return 0;
}

/* ------------------------------------------------------------------------
 * Stochastic prefix verifier (Sec. III-D "Prefix verifier", temperature T>0).
 *
 * The target policy at a row is P = softmax(logits / T).  Request i's
 * candidates are tested in order: candidate x_j = draft[o+j+1] is accepted
 * with probability P_{o+j}(x_j), decided by the caller's uniform u[o+j][0]
 * (accepted iff u < P(x)).  At the first rejection (row o+a) the successor
 * is drawn from P_{o+a} with x_a removed and the rest renormalised; if all
 * k-1 candidates pass, from P_{o+k-1} unchanged.  The draw inverts the
 * cumulative distribution in index order with u[o+a][1]: the successor is
 * the smallest v whose cumulative probability exceeds u.  A candidate id
 * outside [0, vocab) has probability 0 and removes nothing.
 *
 * margin_accept[i] and margin_sample[i] (each may be NULL) receive the
 * smallest distance, in probability, between the request's accept-test
 * uniforms and their thresholds P(x), and between its successor uniform and
 * the nearest boundary of the cumulative distribution it inverts (+inf when
 * there is no such decision): how far the result is from flipping under a
 * perturbation of the probabilities.
 * ---------------------------------------------------------------------- */

/* P(v) for one row: writes prob[0..vocab) (double), returns 0. */
static void row_softmax(const void *logits, int32_t dtype, int64_t base, int32_t vocab,
                        double inv_t, double *prob) {
  double m = -INFINITY;
  for (int32_t v = 0; v < vocab; ++v) {
    double x = logit_at(logits, dtype, base + v) * inv_t;
    if (x > m) m = x;
  }
  double z = 0.0;
  for (int32_t v = 0; v < vocab; ++v) {
    prob[v] = exp(logit_at(logits, dtype, base + v) * inv_t - m);
    z += prob[v];
  }
  for (int32_t v = 0; v < vocab; ++v) prob[v] /= z;
}

int oracle_accept_stochastic(const void *logits, int32_t dtype,
                             const int32_t *cu_qlens, const int32_t *draft_tokens,
                             const float *uniforms, double temperature,
                             int32_t *accept_len, int32_t *next_token,
                             double *margin_accept, double *margin_sample,
                             int32_t num_reqs, int32_t cap, int32_t vocab) {
  if (!logits || !cu_qlens || !draft_tokens || !uniforms || !accept_len || !next_token)
    return -1;
  if (num_reqs < 1 || cap < 1 || vocab < 1 || (dtype != 0 && dtype != 1)) return -1;
  if (!(temperature > 0.0) || !isfinite(temperature)) return -1;
  if (cu_qlens[0] != 0 || cu_qlens[num_reqs] > cap) return -1;
  for (int32_t i = 0; i < num_reqs; ++i)
    if (cu_qlens[i + 1] < cu_qlens[i] || cu_qlens[i + 1] - cu_qlens[i] > 64) return -1;
  double inv_t = 1.0 / temperature;
  double *prob = (double *)malloc(sizeof(double) * (size_t)vocab);
  if (!prob) return -1;
  for (int32_t i = 0; i < num_reqs; ++i) {
    int32_t o = cu_qlens[i];
    int32_t k = cu_qlens[i + 1] - o;
    double mg = INFINITY, ms = INFINITY;
    if (k == 0) {
      accept_len[i] = 0;
      next_token[i] = -1;
      if (margin_accept) margin_accept[i] = mg;
      if (margin_sample) margin_sample[i] = ms;
      continue;
    }
    /* accept candidates while the uniform falls below their probability */
    int32_t a = 0;
    int32_t removed = -1;
    while (a < k - 1) {
      row_softmax(logits, dtype, (int64_t)(o + a) * vocab, vocab, inv_t, prob);
      int32_t x = draft_tokens[o + a + 1];
      double px = (x >= 0 && x < vocab) ? prob[x] : 0.0;
      double u = (double)uniforms[2 * (int64_t)(o + a)];
      if (fabs(u - px) < mg) mg = fabs(u - px);
      if (u < px) {
        ++a;
      } else {
        removed = (x >= 0 && x < vocab) ? x : -1;
        break;
      }
    }
    /* successor: P at row o+a, without the rejected candidate if any */
    row_softmax(logits, dtype, (int64_t)(o + a) * vocab, vocab, inv_t, prob);
    double total = 1.0;
    if (removed >= 0) {
      total -= prob[removed];
      prob[removed] = 0.0;
    }
    double us = (double)uniforms[2 * (int64_t)(o + a) + 1];
    double cum = 0.0;
    int32_t pick = -1, last = -1;
    for (int32_t v = 0; v < vocab; ++v) {
      if (prob[v] <= 0.0) continue;
      double before = cum;
      cum += prob[v] / total;
      last = v;
      if (pick < 0 && cum > us) {
        pick = v;
        ms = us - before < cum - us ? us - before : cum - us;
      }
    }
    if (pick < 0) pick = last; /* u at or past the rounded total */
    accept_len[i] = a;
    next_token[i] = pick;
    if (margin_accept) margin_accept[i] = mg;
    if (margin_sample) margin_sample[i] = ms;
  }
  free(prob);
  return 0;
}

int oracle_successor_interval(const void *logits, int32_t dtype, int32_t row,
                              int32_t vocab, int32_t removed, double temperature,
                              int32_t token, double *lo, double *hi) {
  if (!logits || !lo || !hi || row < 0 || vocab < 1 || token < 0 || token >= vocab)
    return -1;
  if (!(temperature > 0.0) || !isfinite(temperature) || (dtype != 0 && dtype != 1)) return -1;
  double *prob = (double *)malloc(sizeof(double) * (size_t)vocab);
  if (!prob) return -1;
  row_softmax(logits, dtype, (int64_t)row * vocab, vocab, 1.0 / temperature, prob);
  double total = 1.0;
  if (removed >= 0 && removed < vocab) {
    total -= prob[removed];
    prob[removed] = 0.0;
  }
  double cum = 0.0;
  for (int32_t v = 0; v < token; ++v) cum += prob[v] / total;
  *lo = cum;
  *hi = cum + prob[token] / total;
  free(prob);
  return 0;
}

/* ------------------------------------------------------------------------
 * Acceptance predictor forward (Sec. III-C, Eq. (5)): a multilayer
 * perceptron with one ReLU hidden layer, in_dim -> hidden -> out_dim (the
 * paper's 1735 -> 64 -> 15).  For each live request i:
 *   h = max(0, features_i . W1 + b1),   predLogits_i = h . W2 + b2,
 * with W1 [in_dim][hidden], W2 [hidden][out_dim] row-major, everything
 * widened to double.  Rows past n_live get zeros.
 * ---------------------------------------------------------------------- */
int oracle_predictor_forward(const float *features, int32_t n_live, int32_t n_rows,
                             const float *w1, const float *b1, const float *w2,
                             const float *b2, int32_t in_dim, int32_t hidden,
                             int32_t out_dim, double *out) {
  if (!features || !w1 || !b1 || !w2 || !b2 || !out) return -1;
  if (n_rows < 1 || n_live < 0 || n_live > n_rows || in_dim < 1 || hidden < 1 || out_dim < 1)
    return -1;
  double *h = (double *)malloc(sizeof(double) * (size_t)hidden);
  if (!h) return -1;
  for (int32_t i = 0; i < n_rows; ++i) {
    double *o = out + (int64_t)i * out_dim;
    if (i >= n_live) {
      for (int32_t j = 0; j < out_dim; ++j) o[j] = 0.0;
      continue;
    }
    const float *f = features + (int64_t)i * in_dim;
    for (int32_t u = 0; u < hidden; ++u) {
      double acc = (double)b1[u];
      for (int32_t k = 0; k < in_dim; ++k) acc += (double)f[k] * (double)w1[(int64_t)k * hidden + u];
      h[u] = acc > 0.0 ? acc : 0.0;
    }
    for (int32_t j = 0; j < out_dim; ++j) {
      double acc = (double)b2[j];
      for (int32_t u = 0; u < hidden; ++u) acc += h[u] * (double)w2[(int64_t)u * out_dim + j];
      o[j] = acc;
    }
  }
  free(h);
  return 0;
}
