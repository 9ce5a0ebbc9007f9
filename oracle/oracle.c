/*
 * oracle.c -- plain fp64 CPU oracle of the verify hot path of block-diffusion
 * speculative decoding (DScale).
 *
 * TEST INFRASTRUCTURE ONLY: only tests/, __graft_entry__.smoke() and the
 * CPU-baseline leg of bench.py load it.  It shares no code, header or table
 * with the HIP library.  Every floating-point step is in double precision;
 * bf16 and fp32 inputs widen to double exactly.
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
