/*
 * oracle_sanitize_driver.c -- runs every function of the fp64 oracle on small
 * cases with known answers, built together with oracle/oracle.c under
 * AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_oracle_sanitized.py).
 * Any out-of-bounds access, use of uninitialised heap, signed overflow or
 * other undefined behaviour aborts the run; any wrong answer returns 1.
 *
 * The answers are closed forms and the paper's worked examples:
 *   attention  one visible key gives that key's V exactly; a constant V
 *              gives the constant; tail rows are zero (Sec. III-D, Eq. (16));
 *   argmax     ties go to the lowest index, -0 equals +0;
 *   accept     a hand-planted prefix (Sec. III-D prefix verifier, greedy);
 *   stochastic the three-token example P = [1/6, 2/6, 3/6] and its exact
 *              successor intervals;
 *   predictor  one-hot weights select single features (Eq. (5));
 *   DVL        the Sec. III-C worked example: seeds [5, 10, 7, 9] against a
 *              budget of 32 grow R1 to [6, 10, 7, 9] with offsets
 *              [0, 6, 16, 23] and end 32 (Eqs. (8)-(11)).
 * Malformed inputs must be refused with -1.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../oracle/oracle.h"

static int failures = 0;

#define CHECK(cond)                                                          \
  do {                                                                       \
    if (!(cond)) {                                                           \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                            \
    }                                                                        \
  } while (0)

/* bf16 bits of a float that bf16 holds exactly */
static uint16_t bf16_of(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return (uint16_t)(u >> 16);
}

static double from_bf16(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* every buffer exactly its size on the heap, so that ASan sees overruns */
static void *alloc(size_t n) {
  void *p = malloc(n ? n : 1);
  if (!p) exit(2);
  return p;
}

static void test_attention(void) {
  enum { B = 3, HQ = 4, HKV = 1, D = 64, PS = 16, PMAX = 3, NP = 4, CAP = 8 };
  /* request 0: ctx 0, k 1 (one visible key); request 1: ctx 20, k 3 over a
   * constant V; request 2: a sentinel (k 0).  Rows 4..7 are tail rows. */
  const int32_t cu[B + 1] = {0, 1, 4, 4};
  const int32_t ctx[B] = {0, 20, 5};
  int32_t *pt = alloc(sizeof(int32_t) * B * PMAX);
  for (int i = 0; i < B * PMAX; ++i) pt[i] = -1;
  pt[0 * PMAX + 0] = 3;                          /* request 0: page 3 */
  pt[1 * PMAX + 0] = 0, pt[1 * PMAX + 1] = 2;    /* request 1: pages 0, 2 */
  const size_t tile = (size_t)PS * D;            /* elements of one K or V tile */
  uint16_t *kv = alloc(sizeof(uint16_t) * NP * 2 * HKV * tile);
  uint32_t lcg = 12345u;
  for (size_t e = 0; e < (size_t)NP * 2 * HKV * tile; ++e) {
    lcg = lcg * 1664525u + 1013904223u;
    kv[e] = bf16_of((float)((int)(lcg >> 20) - 2048) / 1024.0f);
  }
  const float c = 0.375f;
  for (int p = 0; p < 2; ++p) {  /* constant V on request 1's pages 0 and 2 */
    const int page = p == 0 ? 0 : 2;
    uint16_t *v = kv + ((size_t)page * 2 + 1) * HKV * tile;
    for (size_t e = 0; e < tile; ++e) v[e] = bf16_of(c);
  }
  uint16_t *q = alloc(sizeof(uint16_t) * CAP * HQ * D);
  for (int e = 0; e < CAP * HQ * D; ++e) {
    lcg = lcg * 1664525u + 1013904223u;
    q[e] = bf16_of((float)((int)(lcg >> 22) - 512) / 256.0f);
  }
  double *out = alloc(sizeof(double) * CAP * HQ * D);
  CHECK(oracle_verify_attn(q, cu, kv, pt, ctx, out, B, CAP, HQ, HKV, D, PS, PMAX, NP,
                           0.125) == 0);
  /* request 0 row 0: the only key is slot 0 of page 3; its V tile is
   * dim-major, element (slot s, dim d) at d*16 + s */
  const uint16_t *v3 = kv + ((size_t)3 * 2 + 1) * HKV * tile;
  for (int h = 0; h < HQ; ++h)
    for (int d = 0; d < D; ++d) CHECK(out[(0 * HQ + h) * D + d] == from_bf16(v3[d * PS + 0]));
  for (int r = 1; r < 4; ++r)
    for (int e = 0; e < HQ * D; ++e) CHECK(fabs(out[r * HQ * D + e] - c) < 1e-12);
  for (int r = 4; r < CAP; ++r)
    for (int e = 0; e < HQ * D; ++e) CHECK(out[r * HQ * D + e] == 0.0);
  /* malformed: decreasing offsets, a page id outside the pool */
  const int32_t bad_cu[B + 1] = {0, 2, 1, 1};
  CHECK(oracle_verify_attn(q, bad_cu, kv, pt, ctx, out, B, CAP, HQ, HKV, D, PS, PMAX, NP,
                           0.125) == -1);
  pt[1 * PMAX + 1] = NP;
  CHECK(oracle_verify_attn(q, cu, kv, pt, ctx, out, B, CAP, HQ, HKV, D, PS, PMAX, NP,
                           0.125) == -1);
  free(q), free(kv), free(pt), free(out);
}

static void test_argmax_and_accept(void) {
  enum { ROWS = 5, V = 7 };
  float *lg = alloc(sizeof(float) * ROWS * V);
  for (int e = 0; e < ROWS * V; ++e) lg[e] = -1.0f;
  lg[0 * V + 2] = 3.0f;                          /* row 0: 2 */
  lg[1 * V + 4] = 3.0f, lg[1 * V + 1] = 3.0f;    /* row 1: tie -> 1 */
  lg[2 * V + 6] = 0.5f;                          /* row 2: 6 */
  lg[3 * V + 3] = -0.0f, lg[3 * V + 0] = 0.0f;   /* row 3: +0 and -0 tie -> 0 */
  lg[4 * V + 5] = 9.0f;                          /* row 4: 5 */
  int32_t *idx = alloc(sizeof(int32_t) * ROWS);
  CHECK(oracle_row_argmax(lg, 0, ROWS, V, idx) == 0);
  CHECK(idx[0] == 2 && idx[1] == 1 && idx[2] == 6 && idx[3] == 0 && idx[4] == 5);
  /* request 0 = rows 0..2 (anchor + 2 candidates), request 1 = a sentinel,
   * request 2 = row 3 alone (k = 1); row 4 is a tail row */
  const int32_t cu[4] = {0, 3, 3, 4};
  int32_t draft[ROWS] = {9, 2, 5, 0, 0};  /* t_0 = 2 matches draft[1]; t_1 = 1 != draft[2] */
  int32_t a[3], nx[3];
  CHECK(oracle_accept(lg, 0, cu, draft, a, nx, 3, ROWS, V) == 0);
  CHECK(a[0] == 1 && nx[0] == 1);
  CHECK(a[1] == 0 && nx[1] == -1);
  CHECK(a[2] == 0 && nx[2] == 0);
  draft[2] = 1;  /* now both candidates match: a = k - 1 = 2, successor t_2 = 6 */
  CHECK(oracle_accept(lg, 0, cu, draft, a, nx, 3, ROWS, V) == 0);
  CHECK(a[0] == 2 && nx[0] == 6);
  const int32_t bad_cu[4] = {0, 3, 2, 4};
  CHECK(oracle_accept(lg, 0, bad_cu, draft, a, nx, 3, ROWS, V) == -1);
  free(lg), free(idx);
}

static void test_stochastic(void) {
  /* P = [1/6, 2/6, 3/6] on both rows; candidate x = 2 has P(x) = 1/2 */
  float *lg = alloc(sizeof(float) * 6);
  for (int r = 0; r < 2; ++r)
    for (int v = 0; v < 3; ++v) lg[r * 3 + v] = (float)log((double)(v + 1));
  const int32_t cu[2] = {0, 2};
  const int32_t draft[2] = {7, 2};
  float *u = alloc(sizeof(float) * 4);
  int32_t a, t;
  double ma, ms;
  u[0] = 0.4f, u[1] = 0.3f, u[2] = 0.5f, u[3] = 0.3f;  /* accept; successor 1 */
  CHECK(oracle_accept_stochastic(lg, 0, cu, draft, u, 1.0, &a, &t, &ma, &ms, 1, 2, 3) == 0);
  CHECK(a == 1 && t == 1);
  u[0] = 0.6f, u[1] = 0.5f;  /* reject; P without x = [1/3, 2/3]: 0.5 -> token 1 */
  CHECK(oracle_accept_stochastic(lg, 0, cu, draft, u, 1.0, &a, &t, NULL, NULL, 1, 2, 3) == 0);
  CHECK(a == 0 && t == 1);
  double lo, hi;
  CHECK(oracle_successor_interval(lg, 0, 0, 3, 2, 1.0, 1, &lo, &hi) == 0);
  CHECK(fabs(lo - 1.0 / 3.0) < 1e-6 && fabs(hi - 1.0) < 1e-6);
  CHECK(oracle_successor_interval(lg, 0, 1, 3, -1, 1.0, 2, &lo, &hi) == 0);
  CHECK(fabs(lo - 0.5) < 1e-6 && fabs(hi - 1.0) < 1e-6);
  CHECK(oracle_successor_interval(lg, 0, 0, 3, -1, 0.0, 0, &lo, &hi) == -1);
  CHECK(oracle_accept_stochastic(lg, 0, cu, draft, u, -1.0, &a, &t, NULL, NULL, 1, 2, 3) == -1);
  free(lg), free(u);
}

static void test_predictor(void) {
  enum { N = 3, IN = 5, H = 4, OUT = 2 };
  float *f = alloc(sizeof(float) * N * IN), *w1 = alloc(sizeof(float) * IN * H);
  float *b1 = alloc(sizeof(float) * H), *w2 = alloc(sizeof(float) * H * OUT);
  float *b2 = alloc(sizeof(float) * OUT);
  double *out = alloc(sizeof(double) * N * OUT);
  for (int e = 0; e < N * IN; ++e) f[e] = (float)(e + 1);
  memset(w1, 0, sizeof(float) * IN * H);
  w1[2 * H + 1] = 1.0f;  /* hidden 1 = feature 2 */
  for (int j = 0; j < H; ++j) b1[j] = j == 3 ? -5.0f : 0.0f;  /* hidden 3 cut by ReLU */
  memset(w2, 0, sizeof(float) * H * OUT);
  w2[1 * OUT + 0] = 2.0f, w2[3 * OUT + 1] = 7.0f;
  b2[0] = 0.5f, b2[1] = -1.0f;
  CHECK(oracle_predictor_forward(f, 2, N, w1, b1, w2, b2, IN, H, OUT, out) == 0);
  for (int i = 0; i < 2; ++i) {
    CHECK(out[i * OUT + 0] == 2.0 * f[i * IN + 2] + 0.5);
    CHECK(out[i * OUT + 1] == -1.0);
  }
  CHECK(out[2 * OUT + 0] == 0.0 && out[2 * OUT + 1] == 0.0);  /* past the live count */
  CHECK(oracle_predictor_forward(f, 4, N, w1, b1, w2, b2, IN, H, OUT, out) == -1);
  free(f), free(w1), free(b1), free(w2), free(b2), free(out);
}

static void test_dvl(void) {
  enum { N = 4, W = 16, NBS = 6, MBS = W * NBS / 2 };
  /* scores: logit 0 everywhere gives q = [1, 1/2, 1/2, ...], estimate 7.5,
   * seed floor(7.5 + 0.5) = 8 */
  float *pl = alloc(sizeof(float) * N * (W - 1)), *q = alloc(sizeof(float) * N * W);
  float *ell = alloc(sizeof(float) * N);
  int32_t *k0 = alloc(sizeof(int32_t) * N);
  memset(pl, 0, sizeof(float) * N * (W - 1));
  CHECK(oracle_dvl_scores(pl, N, W, q, ell, k0) == 0);
  for (int i = 0; i < N; ++i) {
    CHECK(q[i * W] == 1.0f && q[i * W + 1] == 0.5f && q[i * W + W - 1] == 0.5f);
    CHECK(ell[i] == 7.5f && k0[i] == 8);
  }
  /* the worked example: seeds [5, 10, 7, 9] (31) against a budget of 32;
   * R1's next slot scores highest, so R1 grows by one */
  const int32_t seeds[N] = {5, 10, 7, 9};
  for (int i = 0; i < N; ++i)
    for (int j = 0; j < W; ++j) q[i * W + j] = j == 0 ? 1.0f : 0.95f - 0.01f * (float)j - 0.1f * (float)i;
  int32_t k[N], updates = -1;
  CHECK(oracle_dvl_adjust(q, seeds, N, W, 32, k, &updates) == 0);
  CHECK(k[0] == 6 && k[1] == 10 && k[2] == 7 && k[3] == 9 && updates == 1);
  CHECK(oracle_dvl_adjust(q, seeds, N, W, N * W + 1, k, &updates) == -1);
  /* pack into a bucket of 6 slots (2 sentinels), M_bs = 48 */
  int32_t *tok = alloc(sizeof(int32_t) * NBS * W), *pos = alloc(sizeof(int32_t) * NBS * W);
  int32_t *ref = alloc(sizeof(int32_t) * NBS * W);
  for (int i = 0; i < NBS * W; ++i) tok[i] = 1000 + i, pos[i] = 2000 + i, ref[i] = 3000 + i;
  int32_t kout[NBS], off[NBS + 1];
  int32_t *pt = alloc(sizeof(int32_t) * MBS), *pp = alloc(sizeof(int32_t) * MBS);
  int32_t *pr = alloc(sizeof(int32_t) * MBS);
  CHECK(oracle_dvl_pack(k, N, NBS, W, MBS, tok, pos, ref, kout, off, pt, pp, pr) == 0);
  const int32_t want_off[NBS + 1] = {0, 6, 16, 23, 32, 32, 32};
  for (int i = 0; i <= NBS; ++i) CHECK(off[i] == want_off[i]);
  CHECK(kout[4] == 0 && kout[5] == 0);
  CHECK(pt[6] == tok[1 * W + 0] && pp[15] == pos[1 * W + 9] && pr[31] == ref[3 * W + 8]);
  for (int s = 32; s < MBS; ++s) CHECK(pt[s] == 0 && pp[s] == 0 && pr[s] == ref[0]);
  const int32_t too_many[N] = {16, 16, 16, 16};
  CHECK(oracle_dvl_pack(too_many, N, NBS, W, 40, tok, pos, ref, kout, off, pt, pp, pr) == -1);
  free(pl), free(q), free(ell), free(k0), free(tok), free(pos), free(ref), free(pt), free(pp),
      free(pr);
}

int main(void) {
  test_attention();
  test_argmax_and_accept();
  test_stochastic();
  test_predictor();
  test_dvl();
  if (failures) {
    fprintf(stderr, "%d check(s) failed\n", failures);
    return 1;
  }
  printf("oracle sanitizer driver: all checks passed\n");
  return 0;
}
