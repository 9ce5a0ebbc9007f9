// dsv_internal.h -- types and small device helpers shared by the HIP sources
// of the verify-path library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dsv.h"

namespace dsv {

// MFMA operand / result vector types (v_mfma_f32_16x16x32_bf16: A and B are
// 8 bf16 per lane, C/D are 4 fp32 per lane).
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kPage = DSV_PAGE_SIZE;  // tokens per KV page
constexpr int kMaxQlen = DSV_MAX_QLEN;

// Verify attention: keys per inner step of the stream-K kernel (two pages),
// and the lead-in of virtual keys that its plan puts in front of every
// segment with keys (the cost of starting a piece on it, six blocks).  The
// host's int32 guard on the flattened work counts the lead-in too.
constexpr int kAttnBlockKeys = 32;
constexpr int kAttnLeadKeys = 6 * kAttnBlockKeys;

// -------------------------------------------------------------------------
// verify attention
// -------------------------------------------------------------------------
struct AttnParams {
  const uint16_t *q;          // bf16 [cap][Hq][D]
  const int32_t *cu;          // [B+1]
  const uint16_t *kv;         // bf16 [P][2][Hkv][16*D]
  const int32_t *page_table;  // [B][P_max]
  const int32_t *ctx;         // [B]
  uint16_t *out;              // bf16 [cap][Hq][D]
  int32_t *plan;              // [2B+3]: key prefix per request, total, share (minus
                              // the piece cap for the small-batch plan), piece prefix
                              // per request, total
  float2 *part_ml;            // fp32 [grid][2][G*16] x (m, l)   (stream-K partials)
  float *part_o;              // fp32 [grid][2][G*16][D]
  int32_t num_reqs, cap, hq, hkv, group, max_pages, num_pages, max_kv_len;
  int32_t num_wg;     // persistent grid of the stream-K kernel
  int32_t num_cu;     // compute units of the device
  float scale_log2;   // softmax scale * log2(e)
};

// Workspace carve-up shared by the size query and the launcher.
struct AttnWorkspace {
  int32_t grid_cap;  // the largest persistent grid the workspace serves
  size_t plan_off, part_ml_off, part_o_off, total;
};

int32_t attn_grid(const dsv_attn_dims &d);  // launch grid on the current device
int32_t attn_num_cu();                      // compute units of the current device
AttnWorkspace attn_workspace_layout(const dsv_attn_dims &d);
hipError_t launch_verify_attn(const AttnParams &p, int head_dim, hipStream_t s);

// -------------------------------------------------------------------------
// acceptance
// -------------------------------------------------------------------------
constexpr int kAcceptChunk = 8192;  // vocabulary elements per argmax workgroup

struct AcceptWorkspace {
  size_t val_off, idx_off, total;
  int32_t num_chunks;
};
AcceptWorkspace accept_workspace_layout(int32_t cap, int32_t vocab);
void *accept_noalloc_scratch();  // the current device's fixed scratch, or nullptr
hipError_t launch_accept(const void *logits, int dtype, const int32_t *cu,
                         const int32_t *draft, int32_t *accept_len,
                         int32_t *next_token, int32_t num_reqs, int32_t cap,
                         int32_t vocab, float *best_val, int32_t *best_idx,
                         int32_t num_chunks, hipStream_t s);

hipError_t launch_validate(const int32_t *cu, const int32_t *ctx,
                           const int32_t *page_table, const dsv_attn_dims &d,
                           int32_t *err_word, hipStream_t s);

// -------------------------------------------------------------------------
// stochastic acceptance (temperature > 0)
// -------------------------------------------------------------------------
struct SampleWorkspace {
  size_t m_off, s_off, total;
  int32_t num_chunks;
};
SampleWorkspace sample_workspace_layout(int32_t cap, int32_t vocab);
hipError_t launch_accept_stochastic(const void *logits, int dtype, const int32_t *cu,
                                    const int32_t *draft, const float *uniforms,
                                    float scale_log2, int32_t *accept_len,
                                    int32_t *next_token, int32_t num_reqs, int32_t cap,
                                    int32_t vocab, float *stat_m, float *stat_s,
                                    int32_t num_chunks, hipStream_t s);

// -------------------------------------------------------------------------
// acceptance predictor
// -------------------------------------------------------------------------
constexpr int kPredHidden = DSV_PRED_HIDDEN;
size_t predictor_workspace_bytes(int32_t n_bs, int32_t in_dim);
hipError_t launch_predictor(const float *features, const int32_t *num_live, const float *w1,
                            const float *b1, const float *w2, const float *b2, float *out,
                            int32_t n_bs, int32_t in_dim, int32_t out_dim, float *part,
                            hipStream_t s);

// -------------------------------------------------------------------------
// DVL allocation and packing
// -------------------------------------------------------------------------
hipError_t launch_dvl(const float *pred_logits, const int32_t *num_live,
                      const int32_t *tokens, const int32_t *positions,
                      const int32_t *kv_refs, int32_t *k_out, int32_t *cu,
                      int32_t *ptok, int32_t *ppos, int32_t *pref, float *scores,
                      int32_t n_bs, int32_t w, hipStream_t s);

// Kernel kinds of the timing hook (see dsv_timing_start).
enum TimingKind {
  kTimeAttnSplit = 0,
  kTimeAttnCombine = 1,
  kTimeArgmax = 2,
  kTimePrefix = 3,
  kTimeDvl = 4,
  kTimeSampleStats = 5,
  kTimeSampleDraw = 6,
  kTimePredictor = 7
};
// Records a HIP event before (end = false) or after (end = true) a launch
// when timing is on and the stream is not being captured.
void timing_mark(int kind, bool end, hipStream_t s);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace dsv
