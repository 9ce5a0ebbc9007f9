/*
 * dsv.h -- C ABI of the block-diffusion speculative-decoding verify path
 * (DScale, "Scaling Block-Diffusion Speculative Decoding with Adaptive
 * Verification"), built for AMD Instinct MI355X (gfx950).
 *
 * The library exposes the two operations of the target-verification hot path,
 * and the decision step that produces its packed layout:
 *
 *   dsv_verify_attn  ragged, packed verify attention over a paged bf16 GQA KV
 *                    cache (Sec. III-B tile routing, Sec. III-D Eq. (16) row
 *                    validity, and the packed layout of Eqs. (10)-(11));
 *   dsv_accept       greedy acceptance: per-row vocabulary argmax followed by
 *                    the longest-prefix compare against the drafted tokens
 *                    (Sec. III-D "Prefix verifier", greedy case; Sec. I
 *                    definition of accepted tokens);
 *   dsv_accept_stochastic
 *                    the same verifier at temperature > 0: probability-ratio
 *                    acceptance with residual resampling (Sec. III-D);
 *   dsv_predictor_forward
 *                    the acceptance predictor (Eq. (5)) that feeds DVL;
 *   dsv_dvl_allocate_pack
 *                    DVL budget allocation and flat-buffer packing (Sec.
 *                    III-C, Alg. 1, Eqs. (6)-(11)): per-request verify
 *                    lengths under the shared budget, the offsets that
 *                    dsv_verify_attn and dsv_accept read as cu_qlens, and the
 *                    packed token, position and cache-reference rows.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every data pointer is a DEVICE pointer owned by the caller.  The library
 *    keeps no pointer after the call returns and allocates nothing.
 *  - Calls only enqueue work on `hip_stream` (a hipStream_t; NULL = the null
 *    stream).  They never synchronise, never read device memory from the
 *    host and never allocate, so they may be recorded into a hipGraph.  The
 *    caller keeps every buffer alive until the enqueued work has finished.
 *  - Host-known arguments are validated before anything is enqueued; on a
 *    validation failure nothing is enqueued and a negative dsv_status is
 *    returned.  The library never aborts the process.
 *  - Device-resident metadata (cu_qlens, ctx_lens, page_table, draft_tokens)
 *    cannot be validated on the host without a synchronisation.  The kernels
 *    re-check it cheaply: a request whose offsets or lengths break a
 *    precondition below is skipped (its outputs are left untouched); a page
 *    id outside [0, num_pages) is never dereferenced (page 0 is read in its
 *    place, so that request's output is unspecified); no access leaves the
 *    buffers described here.  dsv_validate_metadata reports such violations.
 *  - Notation: B = num_reqs, G = num_q_heads / num_kv_heads (GQA group),
 *    D = head_dim, k_i = cu_qlens[i+1] - cu_qlens[i] = verify length of
 *    request i (1 anchor + k_i - 1 drafted candidates; 0 for a sentinel
 *    request that occupies no rows), W = 16 = block width (anchor + 15).
 */
#ifndef DSV_H
#define DSV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DSV_OK = 0,
  DSV_ERR_NULL = -1,        /* a required pointer is NULL                      */
  DSV_ERR_DIMS = -2,        /* a host-known size is out of range               */
  DSV_ERR_UNSUPPORTED = -3, /* valid but unsupported (head_dim, page size, G)  */
  DSV_ERR_WORKSPACE = -4,   /* workspace NULL, misaligned or too small         */
  DSV_ERR_HIP = -5,         /* a HIP runtime call failed (launch error)        */
  DSV_ERR_TOO_LARGE = -6    /* needs more than the fixed scratch of a          */
                            /* no-allocation entry point                       */
} dsv_status;

typedef enum { DSV_F32 = 0, DSV_BF16 = 1 } dsv_dtype;

/* Largest verify length per request: one anchor plus 15 candidates (Sec. II). */
#define DSV_MAX_QLEN 16
/* Tokens per KV page.  The paper cites paged attention without fixing a page
 * size; the library supports exactly 16. */
#define DSV_PAGE_SIZE 16

/*
 * Dimensions of one verify_attn call.  All fields are host values.
 *
 *  num_reqs          B >= 1, the request bucket N_bs (Eq. (14)); requests with
 *                    k_i = 0 are sentinels (Alg. 1's tail requests).
 *  capacity          packed row capacity M_bs of q_packed / out (Eq. (3)),
 *                    >= 1.  Rows cu_qlens[B] .. capacity-1 are tail rows.
 *  num_q_heads       Hq >= 1.
 *  num_kv_heads      Hkv >= 1, Hq % Hkv == 0, G = Hq / Hkv in {1,2,4,8,16}.
 *  head_dim          D in {64, 128}.
 *  page_size         must be DSV_PAGE_SIZE (16).
 *  max_pages_per_req P_max >= 1, the row stride of page_table.
 *  num_pages         pages in kv_pages; page ids must lie in [0, num_pages).
 *  max_kv_len        an upper bound on ctx_lens[i] + k_i over every call that
 *                    uses the same dims, 1 <= max_kv_len <= P_max * 16.
 *  scale             softmax scale applied to q.k (normally 1/sqrt(D)).
 */
typedef struct {
  int32_t num_reqs;
  int32_t capacity;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  int32_t max_pages_per_req;
  int32_t num_pages;
  int32_t max_kv_len;
  float scale;
} dsv_attn_dims;

/*
 * Workspace bytes dsv_verify_attn needs for `dims` (0 if dims are invalid).
 * The workspace holds the work plan and the fp32 partial results (O, m, l) of
 * the (request, KV head) segments that the persistent grid splits between
 * workgroups: at most two per workgroup of a grid of at most 1024, so its
 * size does not grow with max_kv_len.  It needs no initialisation and its
 * contents after a call are unspecified.  Its address may stay fixed across
 * steps (Eq. (13)), so a captured graph can be replayed.
 */
size_t dsv_verify_attn_workspace_bytes(const dsv_attn_dims *dims);

/*
 * Ragged packed verify attention (Eq. (16); Eqs. (10)-(11) packing).
 *
 * For every request i with k_i > 0, every query head h (KV head g = h / G:
 * consecutive query heads share a KV head), and every row j < k_i:
 *
 *   out[cu_qlens[i]+j][h][:] = softmax_t( scale * q . K_t ) . V_t
 *
 * over the keys t = 0 .. ctx_lens[i] + j, i.e. the whole committed context
 * plus the request's own block up to and including row j (request-local
 * causal masking).  K_t / V_t are read from logical position t of request i:
 * page page_table[i*P_max + t/16], slot t%16.  The block's own K/V (anchor and
 * candidates, the paper's "KV refs") must already sit at positions
 * ctx_lens[i] .. ctx_lens[i]+k_i-1 of the same page table.  Tail rows
 * (cu_qlens[B] .. capacity-1) of `out` are written with zeros.  Positional
 * encoding is already applied to q and K.
 *
 * Layouts (bf16 = IEEE binary32 truncated to its upper 16 bits, stored as
 * uint16; all arrays dense, row-major, no padding):
 *   q_packed    bf16 [capacity][Hq][D]; row cu_qlens[i]+j is block row j of i.
 *   cu_qlens    int32 [B+1], cu_qlens[0] = 0, non-decreasing,
 *               k_i <= DSV_MAX_QLEN, cu_qlens[B] <= capacity.
 *   kv_pages    bf16 [num_pages][2][Hkv][16*D]; [..][0][g] is the K tile and
 *               [..][1][g] the V tile of KV head g in that page:
 *                 K tile: element (slot s, dim d) at ((d/8)*16 + s)*8 + d%8
 *                         (8-element d-chunks, slot-major inside a chunk);
 *                 V tile: element (slot s, dim d) at d*16 + s (d-major).
 *               Each tile is 16*D*2 bytes (4 KiB at D=128).  This is the
 *               format every KV writer (the target's KV-cache append) must
 *               produce; it is not the plain [16][D] row layout.  The V tile
 *               must be d-major because the PV product contracts over keys:
 *               one lane's operand is 8 consecutive keys of one dim, which
 *               a plain tile would spread over 8 rows (transposing it at the
 *               LDS store measured 26% slower at Qwen3-8B shape, B=32); the
 *               K tile's 8-dim chunks measured within 1% of a plain K tile
 *               there and up to 4% faster at smaller batches.
 *   page_table  int32 [B][P_max]; only the first ceil((ctx_i+k_i)/16) entries
 *               of row i are read.
 *   ctx_lens    int32 [B], committed context EXCLUDING the verify block, >= 0,
 *               ctx_i + k_i <= max_kv_len.
 *   out         bf16 [capacity][Hq][D], written (every row).
 *   workspace   >= dsv_verify_attn_workspace_bytes(dims) bytes, 256-byte
 *               aligned.
 * q_packed, kv_pages and out must be 16-byte aligned (every base allocation
 * is); DSV_ERR_UNSUPPORTED otherwise, with nothing enqueued.
 * Precision: q.k products, the softmax and all accumulation are fp32; each
 * softmax weight enters the weighted sum of V as a pair of bf16 values (the
 * weight rounded, then the remainder rounded), about 2^-17 of its value, and
 * the normaliser is the fp32 sum of the weights; `out` is rounded once to
 * bf16 (round-to-nearest-even).  Results are bitwise deterministic for given
 * inputs and do not depend on which physical pages hold the keys.  How the
 * other requests are packed changes a request's result only through the
 * summation order (the work split follows the batch's total work), i.e.
 * within rounding.
 */
int dsv_verify_attn(const void *q_packed, const int32_t *cu_qlens,
                    const void *kv_pages, const int32_t *page_table,
                    const int32_t *ctx_lens, void *out,
                    const dsv_attn_dims *dims, void *workspace,
                    size_t workspace_bytes, void *hip_stream);

/*
 * Workspace bytes dsv_accept needs (0 if the sizes are invalid).  It holds
 * per-(row, vocabulary chunk) maxima; it needs no initialisation.
 */
size_t dsv_accept_workspace_bytes(int32_t capacity, int32_t num_reqs,
                                  int32_t vocab);

/*
 * Greedy acceptance (Sec. III-D "Prefix verifier" at temperature 0, where the
 * target policy is one-hot at its argmax; Sec. I: accepted tokens are the
 * contiguous candidate prefix that the target reproduces, anchor excluded).
 *
 * For every live row r < cu_qlens[B]:  t_r = argmax_v logits_packed[r][v]
 * (exact comparison of the stored values; ties go to the lowest v).
 * For request i with o = cu_qlens[i] and k = k_i:
 *   k == 0:  accept_len[i] = 0, next_token[i] = -1 (sentinel request);
 *   k >= 1:  accept_len[i] = a = the largest m <= k-1 such that
 *            t_{o+j} == draft_tokens[o+j+1] for every j < m;
 *            next_token[i] = t_{o+a} (the successor that anchors the next
 *            step: the target's choice at the first rejection, or after the
 *            last accepted candidate).
 *
 * Layouts:
 *   logits_packed  [capacity][vocab] of `dtype` (DSV_F32 or DSV_BF16), dense;
 *                  values of live rows must be finite (NaN order undefined).
 *   cu_qlens       int32 [B+1], as for dsv_verify_attn (same buffer).
 *   draft_tokens   int32 [capacity]: the packed verify INPUT ids -- the anchor
 *                  at row cu_qlens[i], candidate j at row cu_qlens[i]+j.
 *   accept_len     int32 [B], written.
 *   next_token     int32 [B], written.
 *   workspace      >= dsv_accept_workspace_bytes(...) bytes, 256-byte aligned.
 * Rows at or beyond cu_qlens[B] are never read.  The result is exact.
 */
int dsv_accept(const void *logits_packed, int32_t dtype,
               const int32_t *cu_qlens, const int32_t *draft_tokens,
               int32_t *accept_len, int32_t *next_token, int32_t num_reqs,
               int32_t capacity, int32_t vocab, void *workspace,
               size_t workspace_bytes, void *hip_stream);

/*
 * dsv_accept without a workspace argument, for callers that cannot allocate
 * device memory (code under hipGraph capture that must not call hipMalloc,
 * tight serving loops, harnesses that forbid allocation).  Same arguments,
 * semantics and results as dsv_accept, bit for bit, minus the workspace.
 *
 * Scratch: the per-(row, vocabulary chunk) maxima go to a fixed device
 * array of DSV_ACCEPT_NOALLOC_MAX_BYTES that the library holds on every GPU
 * it runs on until the process ends.  A call needs
 * dsv_accept_workspace_bytes(capacity, num_reqs, vocab) of it (about
 * 8 * capacity * ceil(vocab / 8192) bytes, so 27,594 rows at a 151,936-token
 * vocabulary); a larger call returns DSV_ERR_TOO_LARGE and enqueues nothing.
 * The first call on a device resolves the array's address there (no
 * allocation); the array of the CURRENT device is used, so hip_stream must
 * belong to the current device.  The call allocates nothing, frees nothing
 * and calls no allocating library routine.
 *
 * Every call on one GPU shares that GPU's scratch: calls ordered on one
 * stream are safe, but calls that may overlap on one GPU (several streams or
 * host threads) race and their results are undefined.  The scratch needs no
 * initialisation; its contents after a call are unspecified.
 */
#define DSV_ACCEPT_NOALLOC_MAX_BYTES (4u << 20)
int dsv_accept_noalloc(const void *logits_packed, int32_t dtype,
                       const int32_t *cu_qlens, const int32_t *draft_tokens,
                       int32_t *accept_len, int32_t *next_token, int32_t num_reqs,
                       int32_t capacity, int32_t vocab, void *hip_stream);

/*
 * Stochastic acceptance: the prefix verifier at temperature T > 0 (Sec. III-D
 * "Prefix verifier").  The target policy at packed row r is
 * P_r = softmax(logits[r] / T).  For request i (o = cu_qlens[i], k = k_i >= 1)
 * the candidates x_j = draft_tokens[o+j+1], j = 0 .. k-2, are tested in
 * order: x_j is accepted iff uniforms[o+j][0] < P_{o+j}(x_j); the first
 * rejection stops the prefix.  accept_len[i] = a is the number accepted.  The
 * successor is drawn from row o+a: from P_{o+a} with x_a removed and the rest
 * renormalised if x_a was rejected, from P_{o+k-1} unchanged if every
 * candidate passed; the draw takes the smallest token whose cumulative
 * probability (vocabulary order) exceeds uniforms[o+a][1].  For k = 0:
 * accept_len 0, next_token -1.  Over uniform random uniforms the first
 * emitted token is distributed as P at the anchor row (the verifier is
 * lossless).
 *
 *   logits_packed  [capacity][vocab] fp32 or bf16 (dtype); each live row
 *                  has at least one finite logit; -inf logits are allowed
 *                  (probability 0); NaN and +inf are not.
 *   uniforms       fp32 [capacity][2], values in [0, 1), device; the caller
 *                  draws them (e.g. a counter-based generator on the device).
 *   temperature    host float, > 0 and finite (1/T must be finite).
 *   draft_tokens   candidate ids outside [0, vocab) have probability 0.
 *   workspace      >= dsv_accept_stochastic_workspace_bytes(...) bytes,
 *                  256-byte aligned.
 * Arithmetic is fp32 and deterministic.  Every decision compares a uniform
 * with a threshold; it matches exact arithmetic unless the uniform lies
 * within fp32 rounding of that threshold.  Other arguments and metadata
 * rules as for dsv_accept.
 */
size_t dsv_accept_stochastic_workspace_bytes(int32_t capacity, int32_t num_reqs,
                                             int32_t vocab);
int dsv_accept_stochastic(const void *logits_packed, int32_t dtype,
                          const int32_t *cu_qlens, const int32_t *draft_tokens,
                          const float *uniforms, float temperature,
                          int32_t *accept_len, int32_t *next_token, int32_t num_reqs,
                          int32_t capacity, int32_t vocab, void *workspace,
                          size_t workspace_bytes, void *hip_stream);

/*
 * Debug check of device metadata (the preconditions listed above).  Enqueues
 * one small kernel that writes, into *err_word (device int32), a bit mask of
 * the violated rules (0 = all hold):
 *   1  cu_qlens[0] != 0 or not non-decreasing
 *   2  some k_i > DSV_MAX_QLEN
 *   4  cu_qlens[B] > capacity
 *   8  some ctx_lens[i] < 0 or ctx_i + k_i > max_kv_len
 *  16  a page id that verify_attn would read lies outside [0, num_pages)
 * The caller reads *err_word after synchronising the stream.
 */
int dsv_validate_metadata(const int32_t *cu_qlens, const int32_t *ctx_lens,
                          const int32_t *page_table, const dsv_attn_dims *dims,
                          int32_t *err_word, void *hip_stream);

/*
 * Acceptance predictor forward (Sec. III-C, Eqs. (4)-(5)): for each live
 * request i of a bucket of N_bs slots (the first N live, N read on the
 * device and clamped into [0, N_bs]),
 *   h = relu(features_i . W1 + b1),   pred_logits_i = h . W2 + b2,
 * a perceptron with one ReLU hidden layer of DSV_PRED_HIDDEN units (the
 * paper's 1735 -> 64 -> 15, 112,079 parameters).  Rows i >= N of
 * pred_logits are written as 0; their features are not used (any values,
 * NaN included: the rows lie inside the buffer and may be loaded).
 *
 *   features     fp32 [N_bs][in_dim], device.
 *   W1 [in_dim][64], b1 [64], W2 [64][out_dim], b2 [out_dim]: fp32, row-major,
 *                device.
 *   pred_logits  fp32 [N_bs][out_dim], written; with out_dim = W-1 it is the
 *                pred_logits input of dsv_dvl_allocate_pack.
 *   hidden       must be DSV_PRED_HIDDEN (else DSV_ERR_UNSUPPORTED).
 *   workspace    >= dsv_predictor_workspace_bytes(N_bs, in_dim) bytes,
 *                256-byte aligned (per-slice partial sums; no zeroing needed).
 * fp32 arithmetic in a fixed order: deterministic.  Host limits: 1 <= N_bs
 * <= DSV_DVL_MAX_REQS, 1 <= in_dim <= 2^20, 1 <= out_dim <= 1024.
 */
#define DSV_PRED_HIDDEN 64
size_t dsv_predictor_workspace_bytes(int32_t bucket_reqs, int32_t in_dim);
int dsv_predictor_forward(const float *features, const int32_t *num_live, const float *w1,
                          const float *b1, const float *w2, const float *b2,
                          float *pred_logits, int32_t bucket_reqs, int32_t in_dim,
                          int32_t hidden, int32_t out_dim, void *workspace,
                          size_t workspace_bytes, void *hip_stream);

/*
 * DVL budget allocation and flat-buffer packing (Sec. III-C, Alg. 1), for a
 * captured bucket of N_bs request slots of which the first N are live
 * (1 <= N <= N_bs; the rest are sentinels).  W = block_width (16 in the
 * paper), M_live = W*N/2 live rows, M_bs = W*N_bs/2 rows of capacity (Eq. (3)).
 *
 *  1. Prefix scores (Eq. (6)): q_{i,0} = 1 and q_{i,j} = min(q_{i,j-1},
 *     sigmoid(pred_logits[i][j-1])) for j = 1 .. W-1.
 *  2. Initial lengths (Eq. (7)): the estimate is the sum of q_{i,1..W-1}; the
 *     seed is that estimate plus one half, floored, clipped to [1, W].
 *  3. Budget adjustment (Eqs. (8)-(9)): the gap M_live - sum(seeds) is closed
 *     one slot at a time, growing the request whose next slot q_{i,k_i}
 *     scores highest (k_i < W) or shrinking the one whose last slot
 *     q_{i,k_i-1} scores lowest (k_i > 1).  Ties go to the lowest request
 *     index (the paper leaves them open).  The result is the same as that
 *     one-at-a-time loop, computed here without |gap| serial steps.
 *  4. Offsets (Eq. (10)) and packing (Eq. (11)): row offset_i + j of each
 *     packed field holds field_i[j] for j < k_i.  Sentinel requests get
 *     k = 0 and offset M_live; rows M_live .. M_bs-1 get token 0, position 0
 *     and the cache reference kv_refs[0][0].
 *
 * Precision: each score is the binary32 rounding of the sigmoid evaluated in
 * double precision; the running minimum, the estimate (a binary32 sum in
 * position order) and every comparison act on binary32 values.  The result
 * is deterministic and independent of the launch.
 *
 * Arguments (device pointers unless stated):
 *   pred_logits      fp32 [N_bs][W-1], predictor outputs (Eq. (5)); the
 *                    values in rows of sentinel slots are not used.  A NaN
 *                    logit leaves the running minimum unchanged.
 *   num_live         int32 scalar N, read on the device (so a captured graph
 *                    can replay with another live count); values outside
 *                    [0, N_bs] are clamped into it (N = 0 gives M_live = 0).
 *   tokens, positions, kv_refs
 *                    int32 [N_bs][W], each request's full drafted block
 *                    (anchor first); only rows j < k_i of live requests and
 *                    kv_refs[0][0] are read.
 *   k_out            int32 [N_bs], written: lengths (0 for sentinels).
 *   cu_qlens         int32 [N_bs+1], written: offsets, cu_qlens[N_bs] = M_live.
 *   packed_tokens, packed_positions, packed_kv_refs
 *                    int32 [M_bs] each, written in full.
 *   scores_out       fp32 [N_bs][W] or NULL: the prefix scores (zero rows for
 *                    sentinels).
 *   bucket_reqs      N_bs, host value in [1, DSV_DVL_MAX_REQS].
 *   block_width      W, host value, even, in [2, DSV_MAX_QLEN].
 * One workgroup; no workspace; capturable like every other call.
 */
#define DSV_DVL_MAX_REQS 1024
int dsv_dvl_allocate_pack(const float *pred_logits, const int32_t *num_live,
                          const int32_t *tokens, const int32_t *positions,
                          const int32_t *kv_refs, int32_t *k_out,
                          int32_t *cu_qlens, int32_t *packed_tokens,
                          int32_t *packed_positions, int32_t *packed_kv_refs,
                          float *scores_out, int32_t bucket_reqs,
                          int32_t block_width, void *hip_stream);

/*
 * Graph helpers for the fixed-address replay of Alg. 2 (capture once, replay
 * each step) under the workspace invariant of Eq. (13): while a stream is
 * being captured, dsv_verify_attn / dsv_accept calls (and any other work
 * enqueued on it) are recorded instead of run; the instantiated graph then
 * replays them with the same buffer addresses, whose CONTENTS (lengths,
 * offsets, page tables, q, logits) may change between replays.
 *
 *  dsv_graph_capture_begin  starts capture on `hip_stream` (must not be the
 *                           null stream; thread-local capture mode).
 *  dsv_graph_capture_end    ends capture and instantiates; *graph_exec
 *                           receives an opaque handle owned by the caller
 *                           (NULL on failure).
 *  dsv_graph_replay         enqueues one replay on `hip_stream`.
 *  dsv_graph_destroy        releases the handle.
 * All return a dsv_status.
 */
int dsv_graph_capture_begin(void *hip_stream);
int dsv_graph_capture_end(void *hip_stream, void **graph_exec);
int dsv_graph_replay(void *graph_exec, void *hip_stream);
int dsv_graph_destroy(void *graph_exec);

/*
 * Read-rate probe for measurement harnesses; not part of the verify path.
 * Reads `visits` tiles of 4096 bytes from `buf`, tile order[v] at visit v,
 * with 16-byte loads.  A 4 KiB tile is what the verify attention reads per
 * page and KV head (16 tokens x D = 128 x bf16), so a random order over a
 * pool larger than the 256 MB Infinity Cache measures the read rate that
 * scattered page tiles reach, the ceiling the attention is compared with.
 *
 *   buf        device, 16-byte aligned, buf_tiles * 4096 bytes.
 *   order      device int32 [visits]; an id outside [0, buf_tiles) is read
 *              as nothing (contributes 0).
 *   sink       device uint32 [grid]; workgroup b reads visits
 *              [b*per, (b+1)*per), per = ceil(visits / grid), twelve tiles
 *              in flight at a time, and writes the XOR of every 32-bit word
 *              it read to sink[b].
 *   grid       workgroups of 256 threads, 1 .. 65535.
 *
 * Asynchronous on hip_stream; no allocation.  Returns DSV_ERR_NULL,
 * DSV_ERR_DIMS (buf_tiles, visits or grid out of range), DSV_ERR_UNSUPPORTED
 * (buf not 16-byte aligned) or DSV_ERR_HIP (launch failed).
 */
int dsv_read_probe(const void *buf, int32_t buf_tiles, const int32_t *order,
                   int32_t visits, uint32_t *sink, int32_t grid, void *hip_stream);

/*
 * Kernel timing for measurement harnesses.  After dsv_timing_start(n), the
 * next n kernel launches made by eager (not captured) dsv_verify_attn,
 * dsv_accept, dsv_accept_stochastic, dsv_predictor_forward and
 * dsv_dvl_allocate_pack calls are bracketed by HIP events
 * recorded on the caller's stream.  The events are timing-only (created
 * with hipEventDisableSystemFence): recording them performs no system-scope
 * cache writeback or invalidation, so an interval covers the kernel and
 * not such a fence.  dsv_timing_stop waits for those events,
 * writes per kernel kind the summed milliseconds and the launch count (arrays
 * of DSV_TIMING_KINDS), and turns timing off.  Kinds: 0 attention split
 * kernel, 1 attention combine kernel, 2 vocabulary argmax kernel,
 * 3 prefix-compare kernel, 4 DVL allocate-and-pack kernel, 5 softmax
 * statistics kernel and 6 stochastic draw kernel of dsv_accept_stochastic,
 * 7 the two predictor kernels of dsv_predictor_forward (one span).
 * Not thread-safe against concurrent calls from several host threads.
 */
#define DSV_TIMING_KINDS 8
int dsv_timing_start(int32_t max_launches);
int dsv_timing_stop(float *total_ms, int32_t *launches);
/*
 * Like dsv_timing_stop, but writes every recorded launch in order: ms[n] its
 * duration in milliseconds and kinds[n] its kind, for at most `capacity`
 * launches; *count receives the number written.  Turns timing off.
 */
int dsv_timing_stop_each(float *ms, int32_t *kinds, int32_t capacity, int32_t *count);

/* Static text for a dsv_status value ("unknown status" otherwise). */
const char *dsv_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* DSV_H */
