// attn.hip -- ragged, packed verify attention over a paged bf16 GQA KV cache
// for gfx950 (MI355X).
//
// What it computes (Sec. III-D, Eq. (16); packing of Eqs. (10)-(11)): every
// valid row j < k_i of request i reads packed row cu[i]+j and attends, with
// request-local causal masking, to keys 0 .. ctx_i + j of that request.
//
// How (MI355X design; the paper's A100 kernel is a 16-row tile per
// (request, head), Sec. III-B):
//  * Tiles follow the live rows.  The G query heads that share a KV head are
//    stacked with the block rows into R = G*k_i live rows (row r -> block row
//    r / G, head r % G), cut into ceil(R/16) MFMA row tiles, so one K/V read
//    serves all G heads (GQA sharing) and a request never pays for rows it
//    does not have (Eq. (2)'s padding applies per 16-row tile, not per 128).
//  * Split-KV: workgroup (s, g, i) covers keys [s*C, (s+1)*C) of request i and
//    KV head g; requests with one split write bf16 directly, others leave an
//    fp32 partial (O, m, l) that the combine kernel merges in split order.
//    The plan depends only on the request's own lengths, so results do not
//    depend on how the other requests are packed.
//  * Transposed scores: S^T = K Q^T and O^T = V^T P^T with
//    v_mfma_f32_16x16x32_bf16.  The score tile comes out with one query row
//    per lane column, which is exactly the B-operand layout the PV product
//    needs, so P never crosses lanes; the row max needs two xor shuffles.
//  * Every MFMA operand is one direct global load per lane: the K tile is
//    stored in 8-wide d chunks (a wave reads 1 KiB contiguous per load) and
//    the V tile d-major (each lane reads the 4 consecutive keys it multiplies).
//    One operand buffer per wave, reused in place: the next 32-key block's
//    K is loaded as soon as the score MFMAs have consumed the current K, its
//    V as soon as the PV MFMAs have consumed the current V.
//  * Waves of a workgroup split the keys when a request has few row tiles and
//    merge through LDS at the end; with 4 row tiles each wave owns one.
#include "dsv_internal.h"

#include <math.h>
#include <stdlib.h>

namespace dsv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kBlockKeys = 32;  // keys per inner step (two pages)

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ float shfl_xor_f(float x, int m) {
  return __shfl_xor(x, m, kWave);
}

// Two bf16 -> one uint32 (low half first), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ float bf16_round(float x) {
  __bf16 a = (__bf16)x;
  return (float)a;
}

template <int D>
struct KVRegs {
  uint4 k[2][D / 32];  // [page half][32-wide d chunk]: A operand of S^T
  uint2 v[2][D / 16];  // [page half][16-wide d block]: 4 keys of one d
};

// Request-level metadata after the cheap device-side checks.
struct ReqMeta {
  int q0, k, ctx, len;
  bool ok;
};

__device__ __forceinline__ ReqMeta load_req(const AttnParams &p, int i) {
  ReqMeta r;
  r.q0 = p.cu[i];
  const int q1 = p.cu[i + 1];
  r.k = q1 - r.q0;
  r.ctx = p.ctx[i];
  r.len = r.ctx + r.k;
  r.ok = r.k > 0 && r.k <= kMaxQlen && r.q0 >= 0 && q1 <= p.cap &&
         r.ctx >= 0 && r.len <= p.max_kv_len;
  return r;
}

// Base of the K tile of KV head g in the two pages of the 32-key block at
// t0, or nullptr for a page that holds no key below key_end or whose id is
// out of range (never dereferenced).
template <int D>
__device__ __forceinline__ void block_pages(const AttnParams &p, int i, int g,
                                            int t0, int key_end,
                                            const uint16_t *(&kt)[2]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int t = t0 + 16 * h;
    int pid = -1;
    if (t < key_end) pid = p.page_table[(size_t)i * p.max_pages + (t >> 4)];
    kt[h] = (unsigned)pid < (unsigned)p.num_pages
                ? p.kv + ((size_t)pid * 2 * p.hkv + g) * (size_t)(kPage * D)
                : nullptr;
  }
}

template <int D>
__device__ __forceinline__ void load_k(const uint16_t *const (&kt)[2], int lane,
                                       KVRegs<D> &b) {
  const int kq = lane >> 4, n = lane & 15;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (kt[h]) {
#pragma unroll
      for (int c = 0; c < D / 32; ++c)
        b.k[h][c] = *reinterpret_cast<const uint4 *>(kt[h] + ((4 * c + kq) * 16 + n) * 8);
    } else {
#pragma unroll
      for (int c = 0; c < D / 32; ++c) b.k[h][c] = make_uint4(0, 0, 0, 0);
    }
  }
}

template <int D>
__device__ __forceinline__ void load_v(const AttnParams &p,
                                       const uint16_t *const (&kt)[2], int lane,
                                       KVRegs<D> &b) {
  const int kq = lane >> 4, n = lane & 15;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (kt[h]) {
      const uint16_t *vt = kt[h] + (size_t)p.hkv * kPage * D;  // V plane
#pragma unroll
      for (int e = 0; e < D / 16; ++e)
        b.v[h][e] = *reinterpret_cast<const uint2 *>(vt + (16 * e + n) * 16 + 4 * kq);
    } else {
#pragma unroll
      for (int e = 0; e < D / 16; ++e) b.v[h][e] = make_uint2(0, 0);
    }
  }
}

// Online-softmax state of one lane: one query row (lane & 15), the 4 output
// dims 16e + 4*(lane>>4) + [0..3] of each 16-wide d block e.
template <int D>
struct RowState {
  float m, l;
  f32x4 o[D / 16];
};

// Runs one (row tile, key part) item of a split: keys [key_begin, key_end),
// blocks kp, kp + kparts, ... of 32 keys.  One operand buffer: the next
// block's K is loaded as soon as the score MFMAs have consumed the current
// K, and its V as soon as the PV MFMAs have consumed the current V, so each
// load overlaps the math of the other half of the step.
template <int D>
__device__ __forceinline__ void run_item(const AttnParams &p, int i, int g,
                                         const ReqMeta &rq, int rt, int kp,
                                         int kparts, int key_begin, int key_end,
                                         int lane, RowState<D> &st) {
  const int kq = lane >> 4, n = lane & 15;
  const int rows = p.group * rq.k;
  const int rr = rt * 16 + n;
  const bool valid_row = rr < rows;
  const int lg = __builtin_ctz(p.group);
  const int j = rr >> lg, hh = rr & (p.group - 1);
  const int row_limit = valid_row ? rq.ctx + j : -1;

  bf16x8 qv[D / 32];
  {
    const uint16_t *qrow =
        p.q + ((size_t)(rq.q0 + j) * p.hq + (size_t)g * p.group + hh) * D;
#pragma unroll
    for (int c = 0; c < D / 32; ++c) {
      uint4 x = make_uint4(0, 0, 0, 0);
      if (valid_row) x = *reinterpret_cast<const uint4 *>(qrow + 32 * c + 8 * kq);
      qv[c] = as_bf16x8(x);
    }
  }
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int e = 0; e < D / 16; ++e) st.o[e] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nb = (key_end - key_begin + kBlockKeys - 1) / kBlockKeys;
  if (kp >= nb) {
    st.l = 0.f;
    return;
  }
  KVRegs<D> r;
  const uint16_t *kt[2];
  block_pages<D>(p, i, g, key_begin + kp * kBlockKeys, key_end, kt);
  load_k<D>(kt, lane, r);
  load_v<D>(p, kt, lane, r);
  for (int b = kp; b < nb; b += kparts) {
    const int t0 = key_begin + b * kBlockKeys;
    const bool more = b + kparts < nb;
    // --- scores S^T = K Q^T: lane holds keys t0 + 16h + 4kq + [0..3] of its row
    f32x4 s[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      s[h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < D / 32; ++c)
        s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(r.k[h][c]), qv[c],
                                                       s[h], 0, 0, 0);
    }
    const uint16_t *kn[2] = {nullptr, nullptr};
    if (more) {
      block_pages<D>(p, i, g, t0 + kparts * kBlockKeys, key_end, kn);
      load_k<D>(kn, lane, r);
    }
    // --- online softmax (base 2, scale folded in)
    float sc[2][4];
    float bmax = -INFINITY;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = t0 + 16 * h + 4 * kq + q;
        const bool vis = t <= row_limit && t < key_end;
        sc[h][q] = vis ? s[h][q] * p.scale_log2 : -INFINITY;
        bmax = fmaxf(bmax, sc[h][q]);
      }
    bmax = fmaxf(bmax, shfl_xor_f(bmax, 16));
    bmax = fmaxf(bmax, shfl_xor_f(bmax, 32));
    const float m_new = fmaxf(st.m, bmax);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(st.m - m_use);
    // P in bf16 (the PV operand); the row sum uses the same rounded weights
    // so the normalisation matches what multiplies V.
    uint32_t pk[4];
    float psum = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float p0 = bf16_round(exp2f(sc[h][0] - m_use));
      const float p1 = bf16_round(exp2f(sc[h][1] - m_use));
      const float p2 = bf16_round(exp2f(sc[h][2] - m_use));
      const float p3 = bf16_round(exp2f(sc[h][3] - m_use));
      psum += (p0 + p1) + (p2 + p3);
      pk[2 * h] = pack_bf16x2(p0, p1);
      pk[2 * h + 1] = pack_bf16x2(p2, p3);
    }
    st.l = st.l * alpha + psum;
    st.m = m_new;
    const bf16x8 pb = as_bf16x8(make_uint4(pk[0], pk[1], pk[2], pk[3]));
    // --- O^T += V^T P^T.  Keys at or past key_end may hold anything (even
    // NaN): zero their V so that 0 * V stays 0 inside the MFMA.
    uint32_t vmask[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int tb = t0 + 16 * h + 4 * kq;
      vmask[h][0] = (tb + 0 < key_end ? 0x0000FFFFu : 0u) | (tb + 1 < key_end ? 0xFFFF0000u : 0u);
      vmask[h][1] = (tb + 2 < key_end ? 0x0000FFFFu : 0u) | (tb + 3 < key_end ? 0xFFFF0000u : 0u);
    }
    const bool tail = t0 + kBlockKeys > key_end;
#pragma unroll
    for (int e = 0; e < D / 16; ++e) {
      uint2 v0 = r.v[0][e], v1 = r.v[1][e];
      if (tail) {
        v0.x &= vmask[0][0];
        v0.y &= vmask[0][1];
        v1.x &= vmask[1][0];
        v1.y &= vmask[1][1];
      }
      const bf16x8 va = as_bf16x8(make_uint4(v0.x, v0.y, v1.x, v1.y));
      st.o[e] *= alpha;
      st.o[e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, st.o[e], 0, 0, 0);
    }
    if (more) load_v<D>(p, kn, lane, r);
  }
  // the lane holds a partial row sum over its own keys; complete it
  st.l += shfl_xor_f(st.l, 16);
  st.l += shfl_xor_f(st.l, 32);
}

template <int D>
__device__ __forceinline__ void write_item(const AttnParams &p, int g, int s,
                                           int n_splits, const ReqMeta &rq,
                                           int rt, int lane,
                                           const RowState<D> &st) {
  const int kq = lane >> 4, n = lane & 15;
  const int rr = rt * 16 + n;
  if (rr >= p.group * rq.k) return;
  const int lg = __builtin_ctz(p.group);
  const int j = rr >> lg, hh = rr & (p.group - 1);
  const size_t row = (size_t)(rq.q0 + j) * p.hq + (size_t)g * p.group + hh;
  if (n_splits == 1) {
    const float inv = 1.f / st.l;
    uint16_t *o = p.out + row * D + 4 * kq;
#pragma unroll
    for (int e = 0; e < D / 16; ++e) {
      uint2 w;
      w.x = pack_bf16x2(st.o[e][0] * inv, st.o[e][1] * inv);
      w.y = pack_bf16x2(st.o[e][2] * inv, st.o[e][3] * inv);
      *reinterpret_cast<uint2 *>(o + 16 * e) = w;
    }
  } else {
    const size_t prow = (size_t)s * p.cap * p.hq + row;
    float *o = p.part_o + prow * D + 4 * kq;
#pragma unroll
    for (int e = 0; e < D / 16; ++e)
      *reinterpret_cast<f32x4 *>(o + 16 * e) = st.o[e];
    if (kq == 0) p.part_ml[prow] = make_float2(st.m, st.l);
  }
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_split_kernel(AttnParams p) {
  constexpr int kLdsStride = D + 4;  // floats per row; +4 spreads LDS banks
  __shared__ float lds_o[kWaves][16][kLdsStride];
  __shared__ float lds_m[kWaves][16];
  __shared__ float lds_l[kWaves][16];

  const int s = blockIdx.x, g = blockIdx.y, i = blockIdx.z;
  const ReqMeta rq = load_req(p, i);
  if (!rq.ok) return;
  const int key_begin = s * p.chunk;
  if (key_begin >= rq.len) return;
  const int key_end = min(rq.len, key_begin + p.chunk);
  const int n_splits = (rq.len + p.chunk - 1) / p.chunk;

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nt = (p.group * rq.k + 15) / 16;  // live 16-row tiles, 1..16
  // Work split across the 4 waves (uniform over the workgroup):
  //   nt >= 3: wave w owns row tiles w, w+4, ... over all keys of the split;
  //   nt <= 2: 4/nt waves share one row tile, each taking every (4/nt)-th
  //            32-key block, and merge through LDS.
  const int kparts = nt <= 2 ? kWaves / nt : 1;
  const int kp = nt <= 2 ? wave / nt : 0;
  const int rt0 = nt <= 2 ? wave % nt : wave;

  RowState<D> st;
  for (int rt = rt0; rt < nt; rt += kWaves) {
    run_item<D>(p, i, g, rq, rt, kp, kparts, key_begin, key_end, lane, st);
    if (kparts == 1) write_item<D>(p, g, s, n_splits, rq, rt, lane, st);
    if (kparts > 1) break;  // exactly one item per wave when merging
  }
  if (kparts == 1) return;

  const int kq = lane >> 4, n = lane & 15;
  const int slot = kp * nt + rt0;
  if (kp > 0) {
#pragma unroll
    for (int e = 0; e < D / 16; ++e)
      *reinterpret_cast<f32x4 *>(&lds_o[slot][n][16 * e + 4 * kq]) = st.o[e];
    if (kq == 0) {
      lds_m[slot][n] = st.m;
      lds_l[slot][n] = st.l;
    }
  }
  __syncthreads();
  if (kp != 0) return;
  float mx = st.m;
  for (int q = 1; q < kparts; ++q) mx = fmaxf(mx, lds_m[q * nt + rt0][n]);
  const float m_use = mx == -INFINITY ? 0.f : mx;
  const float w0 = exp2f(st.m - m_use);
  st.l *= w0;
#pragma unroll
  for (int e = 0; e < D / 16; ++e) st.o[e] *= w0;
  for (int q = 1; q < kparts; ++q) {
    const int sl = q * nt + rt0;
    const float w = exp2f(lds_m[sl][n] - m_use);
    st.l += w * lds_l[sl][n];
#pragma unroll
    for (int e = 0; e < D / 16; ++e)
      st.o[e] += w * *reinterpret_cast<const f32x4 *>(&lds_o[sl][n][16 * e + 4 * kq]);
  }
  st.m = mx;
  write_item<D>(p, g, s, n_splits, rq, rt0, lane, st);
}

// Merges the split partials of requests with more than one split (fixed
// split order, so the result is deterministic) and zeroes the tail rows.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(AttnParams p) {
  const int g = blockIdx.x, i = blockIdx.y;
  const int G = p.group;
  if (i == p.num_reqs) {
    const int live = min(max(p.cu[p.num_reqs], 0), p.cap);
    const int per_row = G * (D / 8);
    const int total = (p.cap - live) * per_row;
    for (int idx = threadIdx.x; idx < total; idx += kThreads) {
      const int r = live + idx / per_row, rem = idx % per_row;
      const int hh = rem / (D / 8), d8 = rem % (D / 8);
      uint16_t *o = p.out + ((size_t)r * p.hq + (size_t)g * G + hh) * D + 8 * d8;
      *reinterpret_cast<uint4 *>(o) = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  const ReqMeta rq = load_req(p, i);
  if (!rq.ok) return;
  const int n_splits = (rq.len + p.chunk - 1) / p.chunk;
  if (n_splits <= 1) return;
  const int lg = __builtin_ctz(G);
  const int rows = G * rq.k;
  const size_t split_stride = (size_t)p.cap * p.hq;
  for (int idx = threadIdx.x; idx < rows * (D / 4); idx += kThreads) {
    const int rr = idx / (D / 4), d4 = idx % (D / 4);
    const int j = rr >> lg, hh = rr & (G - 1);
    const size_t row = (size_t)(rq.q0 + j) * p.hq + (size_t)g * G + hh;
    float mx = -INFINITY;
    for (int s = 0; s < n_splits; ++s) mx = fmaxf(mx, p.part_ml[s * split_stride + row].x);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float den = 0.f;
    for (int s = 0; s < n_splits; ++s) {
      const float2 ml = p.part_ml[s * split_stride + row];
      const float w = exp2f(ml.x - mx);
      den += w * ml.y;
      acc += w * *reinterpret_cast<const f32x4 *>(p.part_o + (s * split_stride + row) * D + 4 * d4);
    }
    const float inv = 1.f / den;
    uint2 w2;
    w2.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    w2.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *reinterpret_cast<uint2 *>(p.out + row * D + 4 * d4) = w2;
  }
}

int env_chunk() {
  static int v = [] {
    const char *e = getenv("DSV_SPLIT_CHUNK");
    if (!e) return 0;
    int c = atoi(e);
    if (c < kBlockKeys) return 0;
    return c / kBlockKeys * kBlockKeys;
  }();
  return v;
}

}  // namespace

// Keys per split.  Smallest power of two >= 128 for which the split grid
// (requests x KV heads x splits at max_kv_len) stays within 8192 workgroups:
// enough workgroups to fill 256 CUs several times over when contexts are
// ragged, few enough that the fp32 partials stay small next to the KV bytes.
int32_t attn_split_chunk(const dsv_attn_dims &d) {
  const int e = env_chunk();
  if (e > 0) return e;
  const long long heads = (long long)d.num_reqs * d.num_kv_heads;
  int32_t c = 128;
  while (c < 4096 && heads * ((d.max_kv_len + c - 1) / c) > 8192) c *= 2;
  return c;
}

AttnWorkspace attn_workspace_layout(const dsv_attn_dims &d) {
  const int32_t chunk = attn_split_chunk(d);
  const size_t splits = (size_t)((d.max_kv_len + chunk - 1) / chunk);
  const size_t rows = splits * (size_t)d.capacity * d.num_q_heads;
  AttnWorkspace w;
  w.part_o_off = 0;
  w.part_ml_off = align_up(rows * d.head_dim * sizeof(float), 256);
  w.total = align_up(w.part_ml_off + rows * sizeof(float2), 256);
  return w;
}

hipError_t launch_verify_attn(const AttnParams &p, int head_dim, hipStream_t s) {
  const dim3 grid_main(p.num_splits, p.hkv, p.num_reqs);
  const dim3 grid_comb(p.hkv, p.num_reqs + 1);
  timing_mark(kTimeAttnSplit, false, s);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_split_kernel<128>, grid_main, dim3(kThreads), 0, s, p);
  else
    hipLaunchKernelGGL(attn_split_kernel<64>, grid_main, dim3(kThreads), 0, s, p);
  timing_mark(kTimeAttnSplit, true, s);
  timing_mark(kTimeAttnCombine, false, s);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_combine_kernel<128>, grid_comb, dim3(kThreads), 0, s, p);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, grid_comb, dim3(kThreads), 0, s, p);
  timing_mark(kTimeAttnCombine, true, s);
  return hipGetLastError();
}

}  // namespace dsv
