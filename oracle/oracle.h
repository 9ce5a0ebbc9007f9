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

#endif
