// abi.hip -- the extern "C" entry points of libdsv: host-side validation,
// workspace carve-up, launch, and the metadata validator / graph helpers.
#include "dsv_internal.h"

#include <math.h>

#include <cmath>

using namespace dsv;

namespace {

bool aligned256(const void *p) { return ((uintptr_t)p & 255u) == 0; }

bool is_pow2_group(int g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

// Host-known checks shared by the size query, the launcher and the validator.
int check_dims(const dsv_attn_dims *d) {
  if (!d) return DSV_ERR_NULL;
  if (d->num_reqs < 1 || d->num_reqs > 65535 || d->capacity < 1 ||
      d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_kv_heads > 65535 ||
      d->max_pages_per_req < 1 || d->num_pages < 1 || d->max_kv_len < 1)
    return DSV_ERR_DIMS;
  if (d->num_q_heads % d->num_kv_heads != 0) return DSV_ERR_DIMS;
  if ((long long)d->max_kv_len > (long long)d->max_pages_per_req * DSV_PAGE_SIZE)
    return DSV_ERR_DIMS;
  if (!(d->scale > 0.f) || !isfinite(d->scale)) return DSV_ERR_DIMS;
  // the flattened work (KV heads x requests x keys, each segment after its
  // stream-K lead-in) is indexed with int32
  const long long seg_keys =
      (long long)(d->max_kv_len + kAttnBlockKeys - 1) / kAttnBlockKeys * kAttnBlockKeys +
      kAttnLeadKeys;
  if ((long long)d->num_kv_heads * d->num_reqs * seg_keys >= (1LL << 30)) return DSV_ERR_DIMS;
  if (d->page_size != DSV_PAGE_SIZE) return DSV_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return DSV_ERR_UNSUPPORTED;
  if (!is_pow2_group(d->num_q_heads / d->num_kv_heads)) return DSV_ERR_UNSUPPORTED;
  return DSV_OK;
}

__global__ void validate_kernel(const int32_t *cu, const int32_t *ctx,
                                const int32_t *page_table, dsv_attn_dims d,
                                int32_t *err_word) {
  __shared__ int32_t err;
  if (threadIdx.x == 0) err = 0;
  __syncthreads();
  int32_t mine = 0;
  if (threadIdx.x == 0 && cu[0] != 0) mine |= 1;
  if (threadIdx.x == 0 && cu[d.num_reqs] > d.capacity) mine |= 4;
  for (int i = threadIdx.x; i < d.num_reqs; i += blockDim.x) {
    const int k = cu[i + 1] - cu[i];
    if (k < 0) mine |= 1;
    if (k > DSV_MAX_QLEN) mine |= 2;
    const long long len = (long long)ctx[i] + (k > 0 ? k : 0);
    if (ctx[i] < 0 || len > d.max_kv_len) mine |= 8;
    if (k > 0 && ctx[i] >= 0 && len <= (long long)d.max_pages_per_req * DSV_PAGE_SIZE) {
      const int pages = (int)((len + DSV_PAGE_SIZE - 1) / DSV_PAGE_SIZE);
      for (int q = 0; q < pages; ++q) {
        const int pid = page_table[(size_t)i * d.max_pages_per_req + q];
        if (pid < 0 || pid >= d.num_pages) mine |= 16;
      }
    }
  }
  if (mine) atomicOr(&err, mine);
  __syncthreads();
  if (threadIdx.x == 0) *err_word = err;
}

}  // namespace

extern "C" {

size_t dsv_verify_attn_workspace_bytes(const dsv_attn_dims *dims) {
  if (check_dims(dims) != DSV_OK) return 0;
  return attn_workspace_layout(*dims).total;
}

int dsv_verify_attn(const void *q_packed, const int32_t *cu_qlens,
                    const void *kv_pages, const int32_t *page_table,
                    const int32_t *ctx_lens, void *out,
                    const dsv_attn_dims *dims, void *workspace,
                    size_t workspace_bytes, void *hip_stream) {
  if (!q_packed || !cu_qlens || !kv_pages || !page_table || !ctx_lens || !out)
    return DSV_ERR_NULL;
  const int rc = check_dims(dims);
  if (rc != DSV_OK) return rc;
  // q rows, K/V tiles and out rows move in 16-byte vectors
  if (((uintptr_t)q_packed | (uintptr_t)kv_pages | (uintptr_t)out) & 15u)
    return DSV_ERR_UNSUPPORTED;
  const AttnWorkspace ws = attn_workspace_layout(*dims);
  if (!workspace || !aligned256(workspace) || workspace_bytes < ws.total)
    return DSV_ERR_WORKSPACE;
  const int32_t grid = attn_grid(*dims);
  if (grid <= 0) return DSV_ERR_HIP;  // device query failed

  AttnParams p;
  p.q = (const uint16_t *)q_packed;
  p.cu = cu_qlens;
  p.kv = (const uint16_t *)kv_pages;
  p.page_table = page_table;
  p.ctx = ctx_lens;
  p.out = (uint16_t *)out;
  p.plan = (int32_t *)((char *)workspace + ws.plan_off);
  p.part_ml = (float2 *)((char *)workspace + ws.part_ml_off);
  p.part_o = (float *)((char *)workspace + ws.part_o_off);
  p.num_reqs = dims->num_reqs;
  p.cap = dims->capacity;
  p.hq = dims->num_q_heads;
  p.hkv = dims->num_kv_heads;
  p.group = dims->num_q_heads / dims->num_kv_heads;
  p.max_pages = dims->max_pages_per_req;
  p.num_pages = dims->num_pages;
  p.max_kv_len = dims->max_kv_len;
  p.num_wg = grid;
  p.num_cu = attn_num_cu();
  if (p.num_cu <= 0) return DSV_ERR_HIP;  // device query failed
  p.scale_log2 = dims->scale * 1.4426950408889634f;
  const hipError_t e = launch_verify_attn(p, dims->head_dim, (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

size_t dsv_accept_workspace_bytes(int32_t capacity, int32_t num_reqs, int32_t vocab) {
  if (capacity < 1 || capacity > 65535 || num_reqs < 1 || vocab < 1) return 0;
  return accept_workspace_layout(capacity, vocab).total;
}

int dsv_accept(const void *logits_packed, int32_t dtype, const int32_t *cu_qlens,
               const int32_t *draft_tokens, int32_t *accept_len,
               int32_t *next_token, int32_t num_reqs, int32_t capacity,
               int32_t vocab, void *workspace, size_t workspace_bytes,
               void *hip_stream) {
  if (!logits_packed || !cu_qlens || !draft_tokens || !accept_len || !next_token)
    return DSV_ERR_NULL;
  if (num_reqs < 1 || capacity < 1 || vocab < 1 || capacity > 65535 ||
      num_reqs > (1 << 30))
    return DSV_ERR_DIMS;
  if (dtype != DSV_F32 && dtype != DSV_BF16) return DSV_ERR_UNSUPPORTED;
  const AcceptWorkspace ws = accept_workspace_layout(capacity, vocab);
  if (!workspace || !aligned256(workspace) || workspace_bytes < ws.total)
    return DSV_ERR_WORKSPACE;
  const hipError_t e = launch_accept(
      logits_packed, dtype, cu_qlens, draft_tokens, accept_len, next_token,
      num_reqs, capacity, vocab, (float *)((char *)workspace + ws.val_off),
      (int32_t *)((char *)workspace + ws.idx_off), ws.num_chunks,
      (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

int dsv_accept_noalloc(const void *logits_packed, int32_t dtype, const int32_t *cu_qlens,
                       const int32_t *draft_tokens, int32_t *accept_len,
                       int32_t *next_token, int32_t num_reqs, int32_t capacity,
                       int32_t vocab, void *hip_stream) {
  if (!logits_packed || !cu_qlens || !draft_tokens || !accept_len || !next_token)
    return DSV_ERR_NULL;
  if (num_reqs < 1 || capacity < 1 || vocab < 1 || capacity > 65535 ||
      num_reqs > (1 << 30))
    return DSV_ERR_DIMS;
  if (dtype != DSV_F32 && dtype != DSV_BF16) return DSV_ERR_UNSUPPORTED;
  const AcceptWorkspace ws = accept_workspace_layout(capacity, vocab);
  if (ws.total > DSV_ACCEPT_NOALLOC_MAX_BYTES) return DSV_ERR_TOO_LARGE;
  char *scratch = (char *)accept_noalloc_scratch();
  if (!scratch) return DSV_ERR_HIP;
  const hipError_t e = launch_accept(
      logits_packed, dtype, cu_qlens, draft_tokens, accept_len, next_token,
      num_reqs, capacity, vocab, (float *)(scratch + ws.val_off),
      (int32_t *)(scratch + ws.idx_off), ws.num_chunks, (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

size_t dsv_accept_stochastic_workspace_bytes(int32_t capacity, int32_t num_reqs,
                                             int32_t vocab) {
  if (capacity < 1 || num_reqs < 1 || vocab < 1) return 0;
  return sample_workspace_layout(capacity, vocab).total;
}

int dsv_accept_stochastic(const void *logits_packed, int32_t dtype, const int32_t *cu_qlens,
                          const int32_t *draft_tokens, const float *uniforms,
                          float temperature, int32_t *accept_len, int32_t *next_token,
                          int32_t num_reqs, int32_t capacity, int32_t vocab,
                          void *workspace, size_t workspace_bytes, void *hip_stream) {
  if (!logits_packed || !cu_qlens || !draft_tokens || !uniforms || !accept_len ||
      !next_token)
    return DSV_ERR_NULL;
  if (num_reqs < 1 || capacity < 1 || vocab < 1 || capacity > 65535 ||
      num_reqs > (1 << 30))
    return DSV_ERR_DIMS;
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return DSV_ERR_DIMS;
  const float scale_log2 = (float)(1.4426950408889634 / (double)temperature);
  if (!std::isfinite(scale_log2)) return DSV_ERR_DIMS;
  if (dtype != DSV_F32 && dtype != DSV_BF16) return DSV_ERR_UNSUPPORTED;
  const SampleWorkspace ws = sample_workspace_layout(capacity, vocab);
  if (!workspace || !aligned256(workspace) || workspace_bytes < ws.total)
    return DSV_ERR_WORKSPACE;
  const hipError_t e = launch_accept_stochastic(
      logits_packed, dtype, cu_qlens, draft_tokens, uniforms, scale_log2, accept_len,
      next_token, num_reqs, capacity, vocab, (float *)((char *)workspace + ws.m_off),
      (float *)((char *)workspace + ws.s_off), ws.num_chunks, (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

int dsv_validate_metadata(const int32_t *cu_qlens, const int32_t *ctx_lens,
                          const int32_t *page_table, const dsv_attn_dims *dims,
                          int32_t *err_word, void *hip_stream) {
  if (!cu_qlens || !ctx_lens || !page_table || !err_word) return DSV_ERR_NULL;
  const int rc = check_dims(dims);
  if (rc != DSV_OK) return rc;
  hipLaunchKernelGGL(validate_kernel, dim3(1), dim3(256), 0, (hipStream_t)hip_stream,
                     cu_qlens, ctx_lens, page_table, *dims, err_word);
  return hipGetLastError() == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

size_t dsv_predictor_workspace_bytes(int32_t bucket_reqs, int32_t in_dim) {
  if (bucket_reqs < 1 || bucket_reqs > DSV_DVL_MAX_REQS || in_dim < 1 || in_dim > (1 << 20))
    return 0;
  return predictor_workspace_bytes(bucket_reqs, in_dim);
}

int dsv_predictor_forward(const float *features, const int32_t *num_live, const float *w1,
                          const float *b1, const float *w2, const float *b2,
                          float *pred_logits, int32_t bucket_reqs, int32_t in_dim,
                          int32_t hidden, int32_t out_dim, void *workspace,
                          size_t workspace_bytes, void *hip_stream) {
  if (!features || !num_live || !w1 || !b1 || !w2 || !b2 || !pred_logits) return DSV_ERR_NULL;
  if (bucket_reqs < 1 || bucket_reqs > DSV_DVL_MAX_REQS || in_dim < 1 || in_dim > (1 << 20) ||
      out_dim < 1 || out_dim > 1024)
    return DSV_ERR_DIMS;
  if (hidden != DSV_PRED_HIDDEN) return DSV_ERR_UNSUPPORTED;
  if (!workspace || !aligned256(workspace) ||
      workspace_bytes < predictor_workspace_bytes(bucket_reqs, in_dim))
    return DSV_ERR_WORKSPACE;
  const hipError_t e = launch_predictor(features, num_live, w1, b1, w2, b2, pred_logits,
                                        bucket_reqs, in_dim, out_dim, (float *)workspace,
                                        (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

int dsv_dvl_allocate_pack(const float *pred_logits, const int32_t *num_live,
                          const int32_t *tokens, const int32_t *positions,
                          const int32_t *kv_refs, int32_t *k_out,
                          int32_t *cu_qlens, int32_t *packed_tokens,
                          int32_t *packed_positions, int32_t *packed_kv_refs,
                          float *scores_out, int32_t bucket_reqs,
                          int32_t block_width, void *hip_stream) {
  if (!pred_logits || !num_live || !tokens || !positions || !kv_refs || !k_out ||
      !cu_qlens || !packed_tokens || !packed_positions || !packed_kv_refs)
    return DSV_ERR_NULL;
  if (bucket_reqs < 1 || bucket_reqs > DSV_DVL_MAX_REQS) return DSV_ERR_DIMS;
  if (block_width < 2 || block_width > DSV_MAX_QLEN || block_width % 2 != 0)
    return DSV_ERR_DIMS;
  const hipError_t e = launch_dvl(pred_logits, num_live, tokens, positions, kv_refs,
                                  k_out, cu_qlens, packed_tokens, packed_positions,
                                  packed_kv_refs, scores_out, bucket_reqs, block_width,
                                  (hipStream_t)hip_stream);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

int dsv_graph_capture_begin(void *hip_stream) {
  if (!hip_stream) return DSV_ERR_NULL;
  const hipError_t e =
      hipStreamBeginCapture((hipStream_t)hip_stream, hipStreamCaptureModeThreadLocal);
  return e == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}

int dsv_graph_capture_end(void *hip_stream, void **graph_exec) {
  if (!hip_stream || !graph_exec) return DSV_ERR_NULL;
  *graph_exec = nullptr;
  hipGraph_t g = nullptr;
  if (hipStreamEndCapture((hipStream_t)hip_stream, &g) != hipSuccess || !g)
    return DSV_ERR_HIP;
  hipGraphExec_t ex = nullptr;
  const hipError_t e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e != hipSuccess) return DSV_ERR_HIP;
  *graph_exec = (void *)ex;
  return DSV_OK;
}

int dsv_graph_replay(void *graph_exec, void *hip_stream) {
  if (!graph_exec) return DSV_ERR_NULL;
  return hipGraphLaunch((hipGraphExec_t)graph_exec, (hipStream_t)hip_stream) == hipSuccess
             ? DSV_OK
             : DSV_ERR_HIP;
}

int dsv_graph_destroy(void *graph_exec) {
  if (!graph_exec) return DSV_ERR_NULL;
  return hipGraphExecDestroy((hipGraphExec_t)graph_exec) == hipSuccess ? DSV_OK
                                                                       : DSV_ERR_HIP;
}

const char *dsv_status_string(int status) {
  switch (status) {
    case DSV_OK: return "ok";
    case DSV_ERR_NULL: return "null pointer argument";
    case DSV_ERR_DIMS: return "dimension out of range";
    case DSV_ERR_UNSUPPORTED: return "unsupported configuration";
    case DSV_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DSV_ERR_HIP: return "HIP runtime error";
    case DSV_ERR_TOO_LARGE: return "exceeds the fixed scratch of the no-allocation entry point";
    default: return "unknown status";
  }
}

}  // extern "C"
