// attn.hip -- ragged, packed verify attention over a paged bf16 GQA KV cache
// for gfx950 (MI355X).
//
// What it computes (Sec. III-D, Eq. (16); packing of Eqs. (10)-(11)): every
// valid row j < k_i of request i reads packed row cu[i]+j and attends, with
// request-local causal masking, to keys 0 .. ctx_i + j of that request.
//
// How (MI355X design; the paper's A100 kernel is a 16-row tile per
// (request, head) on a grid of requests x heads, Sec. III-B):
//  * Tiles follow the live rows.  The G query heads that share a KV head are
//    stacked with the block rows into R = G*k_i live rows (row r -> block row
//    r / G, head r % G), cut into ceil(R/16) MFMA row tiles, so one K/V read
//    serves all G heads (GQA sharing) and a request never pays for rows it
//    does not have (Eq. (2)'s padding applies per 16-row tile, not per 128).
//  * Stream-K work split.  Each (request, KV head) pair is a segment of
//    ceil32(ctx_i + k_i) keys; the segments are laid end to end and a
//    persistent grid, sized to the workgroups the GPU holds at once, gives
//    every workgroup one equal contiguous share.  A workgroup walks the
//    segments its share touches; a segment it covers whole is written as
//    bf16 directly, a segment cut at a share boundary leaves an fp32 partial
//    (O, m, l) that the combine kernel merges in workgroup order.  Ragged
//    contexts cost no idle workgroups, and there are at most two partials
//    per workgroup.  Results depend only on the request's own data and the
//    batch's total work (the share size), and merge in a fixed order, so
//    they are deterministic.
//  * Transposed scores: S^T = K Q^T and O^T = V^T P^T with
//    v_mfma_f32_16x16x32_bf16.  The score tile comes out with one query row
//    per lane column, which is exactly the B-operand layout the PV product
//    needs, so P never crosses lanes; the row max needs two xor shuffles.
//  * Every MFMA operand is one direct global load per lane: the K tile is
//    stored in 8-wide d chunks (a wave reads 1 KiB contiguous per load) and
//    the V tile d-major (each lane reads the 4 consecutive keys it
//    multiplies).  One operand buffer per wave, reused in place: the next
//    32-key block's K is loaded as soon as the score MFMAs have consumed the
//    current K, its V as soon as the PV MFMAs have consumed the current V.
//    Page ids are fetched 64 at a time into a lane-indexed register and read
//    with v_readlane, so no page-table load sits in front of a K/V load.
//  * Waves of a workgroup split the keys when a request has few row tiles and
//    merge through LDS; with three or more row tiles each wave owns tiles.
#include "dsv_internal.h"

#include <math.h>

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

__device__ __forceinline__ int round_up_block(int x) {
  return (x + kBlockKeys - 1) / kBlockKeys * kBlockKeys;
}

// Request-level metadata after the cheap device-side checks.  `seg` is the
// request's segment length in keys (ctx + k rounded up to 32), 0 for a
// sentinel or a request whose metadata breaks the contract.
struct ReqMeta {
  int q0, k, ctx, len, seg;
};

__device__ __forceinline__ int segment_of(const AttnParams &p, int q0, int q1, int ctx) {
  const int k = q1 - q0;
  const bool ok = k > 0 && k <= kMaxQlen && q0 >= 0 && q1 <= p.cap && ctx >= 0 &&
                  ctx + k <= p.max_kv_len;
  return ok ? round_up_block(ctx + k) : 0;
}

// Per-thread (non-uniform) segment length of request i.
__device__ __forceinline__ int segment_len(const AttnParams &p, int i) {
  return segment_of(p, p.cu[i], p.cu[i + 1], p.ctx[i]);
}

// Uniform metadata of request i: read with vector loads (the kernel writes
// global memory, so the compiler will not use the scalar cache) and then
// declared uniform.
__device__ __forceinline__ ReqMeta load_req(const AttnParams &p, int i) {
  ReqMeta r;
  r.q0 = __builtin_amdgcn_readfirstlane(p.cu[i]);
  const int q1 = __builtin_amdgcn_readfirstlane(p.cu[i + 1]);
  r.ctx = __builtin_amdgcn_readfirstlane(p.ctx[i]);
  r.k = q1 - r.q0;
  r.len = r.ctx + r.k;
  r.seg = segment_of(p, r.q0, q1, r.ctx);
  return r;
}

// ------------------------------------------------------------------ LDS ring
// One 32-key block in LDS holds the MFMA operand tiles of K (two 16-key
// score halves x D/32 chunks of 32 dims) and of V (D/16 blocks of 16 dims),
// 1 KiB each and stored in lane order: lane l's 16 bytes sit at l*16, so a
// wave reads an operand with one conflict-free ds_read_b128 and a ring load
// (global_load_lds_dwordx4, written by each lane at its own slot) fills one.
template <int D>
struct RingShape {
  static constexpr int kKOps = 2 * (D / 32);
  static constexpr int kVOps = D / 16;
  static constexpr int kOps = kKOps + kVOps;          // 16 at D = 128
  static constexpr int kOpsPerWave = kOps / kWaves;   // ring loads per wave per block
};
constexpr int kStages = 4;      // blocks resident in the ring (3 in flight)
constexpr int kSubPages = 128;  // page ids staged in LDS at a time (2048 keys)

// s_waitcnt immediate (gfx9 encoding): wait until at most `vm` vector-memory
// and `lgkm` LDS/scalar operations of this wave are outstanding.
constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 15) | (7 << 4) | ((lgkm & 15) << 8) | (((vm >> 4) & 3) << 14);
}

// Workgroup barrier without the memory fence __syncthreads() adds (that
// fence would drain every ring load in flight); callers wait explicitly for
// what must be complete first.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Ring operand reads.  One inline-asm block issues the ds_read_b128 of all
// K (or all V) operand tiles of a stage and waits for them, so its outputs
// exist only once the data is in registers.  Asm, because the compiler cannot
// tell ring stages apart and would otherwise wait for every ring load in
// flight before each read; the stage read here is complete by construction
// (explicit wait + barrier at the top of the step).  `base` is the LDS
// address of this lane's slot in the stage (stage + lane * 16).
template <int D>
struct RingRead;

template <>
struct RingRead<128> {
  static __device__ __forceinline__ void k(uint32_t base, uint4 (&o)[8]) {
    asm volatile(
        "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
        "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]),
          "=&v"(o[6]), "=&v"(o[7])
        : "v"(base)
        : "memory");
  }
};

template <>
struct RingRead<64> {
  static __device__ __forceinline__ void k(uint32_t base, uint4 (&o)[4]) {
    asm volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %4 offset:1024\n\t"
        "ds_read_b128 %2, %4 offset:2048\n\tds_read_b128 %3, %4 offset:3072\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3])
        : "v"(base)
        : "memory");
  }
};

// The first `n` (1, 2, 4 or 8) V operand tiles starting at LDS address
// `base`, read and waited for in one asm block.
template <int N>
__device__ __forceinline__ void ring_read_v(uint32_t base, uint4 (&o)[8]) {
  if constexpr (N == 1) {
    asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]) : "v"(base) : "memory");
  } else if constexpr (N == 2) {
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:1024\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1]) : "v"(base) : "memory");
  } else if constexpr (N == 4) {
    asm volatile("ds_read_b128 %0, %4\n\tds_read_b128 %1, %4 offset:1024\n\t"
                 "ds_read_b128 %2, %4 offset:2048\n\tds_read_b128 %3, %4 offset:3072\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]) : "v"(base) : "memory");
  } else {
    asm volatile(
        "ds_read_b128 %0, %8\n\tds_read_b128 %1, %8 offset:1024\n\t"
        "ds_read_b128 %2, %8 offset:2048\n\tds_read_b128 %3, %8 offset:3072\n\t"
        "ds_read_b128 %4, %8 offset:4096\n\tds_read_b128 %5, %8 offset:5120\n\t"
        "ds_read_b128 %6, %8 offset:6144\n\tds_read_b128 %7, %8 offset:7168\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]),
          "=&v"(o[6]), "=&v"(o[7])
        : "v"(base)
        : "memory");
  }
}

// Key order inside a block.  Row m of score half hh holds key
// 8*(m/4) + 4*hh + m%4, so after S^T = K Q^T the lane with k-group kq holds
// keys 8*kq + [0..7] of its query row: exactly the order the PV product
// contracts over, and V's operand for that lane is 8 consecutive keys of one
// dim, one 16-byte read of the d-major V tile.
__device__ __forceinline__ int score_key(int hh, int m) { return 8 * (m >> 2) + 4 * hh + (m & 3); }

// Issues this wave's share of the ring loads of one block (pages pid0,
// pid1) into `stage`.  An invalid page id reads the start of the pool
// instead (a valid address); the compute step masks those keys.
template <int D>
__device__ __forceinline__ void ring_load(const AttnParams &p, int g, int pid0, int pid1,
                                          uint4 (*stage)[kWave], int wave, int lane) {
  using R = RingShape<D>;
  const int m = lane & 15, kgrp = lane >> 4;
  const bool ok0 = (unsigned)pid0 < (unsigned)p.num_pages;
  const bool ok1 = (unsigned)pid1 < (unsigned)p.num_pages;
  const size_t tile = (size_t)kPage * D;
  const uint16_t *k0 = p.kv + (ok0 ? ((size_t)pid0 * 2 * p.hkv + g) * tile : 0);
  const uint16_t *k1 = p.kv + (ok1 ? ((size_t)pid1 * 2 * p.hkv + g) * tile : 0);
  const uint16_t *v0 = k0 + (ok0 ? (size_t)p.hkv * tile : 0);
  const uint16_t *v1 = k1 + (ok1 ? (size_t)p.hkv * tile : 0);
#pragma unroll
  for (int u = 0; u < R::kOpsPerWave; ++u) {
    const int op = wave * R::kOpsPerWave + u;
    const uint16_t *src;
    if (op < R::kKOps) {
      const int hh = op / (D / 32), c = op % (D / 32);
      const int key = score_key(hh, m);
      src = (key < 16 ? k0 : k1) + ((4 * c + kgrp) * 16 + (key & 15)) * 8;
    } else {
      const int e = op - R::kKOps;
      src = (kgrp >= 2 ? v1 : v0) + (16 * e + m) * 16 + 8 * (kgrp & 1);
    }
    __builtin_amdgcn_global_load_lds(src, &stage[op][0], 16, 0, 0);
  }
}

// Online-softmax state of one lane: one query row (lane & 15) and, for each
// of the wave's d blocks u (dims 16*(e_lo+u) + 4*(lane>>4) + [0..3]), the 4
// accumulated outputs.
template <int D>
struct RowState {
  float m, l;
  f32x4 o[D / 16];
};

// One 32-key block from the ring: scores for the wave's row tile, online
// softmax, and the PV product for the wave's `ne` d blocks starting at e_lo.
// `full` (uniform) says every key of the block is visible to every live row
// and both pages are valid, so no masking is needed.
template <int D, int NE>
__device__ __forceinline__ void ring_compute(const uint4 (*stage)[kWave], int lane, int t0,
                                             int key_end, int row_limit, bool full, bool ok0,
                                             bool ok1, const bf16x8 (&qv)[D / 32], int e_lo,
                                             float scale_log2, RowState<D> &st) {
  using R = RingShape<D>;
  const int kq = lane >> 4;
  const uint32_t base = (uint32_t)(uintptr_t)&stage[0][lane];  // LDS offset: low half
  uint4 kop[R::kKOps];
  RingRead<D>::k(base, kop);
  f32x4 s[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    s[h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
      s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kop[h * (D / 32) + c]), qv[c],
                                                     s[h], 0, 0, 0);
  }
  // element (h, q) of this lane is key t0 + 8kq + 4h + q, in page kq / 2
  const bool page_ok = kq >= 2 ? ok1 : ok0;
  float sc[2][4];
  if (full) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q) sc[h][q] = s[h][q] * scale_log2;
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = t0 + 8 * kq + 4 * h + q;
        const bool vis = t <= row_limit && t < key_end && page_ok;
        sc[h][q] = vis ? s[h][q] * scale_log2 : -INFINITY;
      }
  }
  float bmax = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                     fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
  bmax = fmaxf(bmax, shfl_xor_f(bmax, 16));
  bmax = fmaxf(bmax, shfl_xor_f(bmax, 32));
  const float m_new = fmaxf(st.m, bmax);
  const float m_use = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = __builtin_amdgcn_exp2f(st.m - m_use);
  // P in bf16 (the PV operand); the row sum uses the same rounded weights so
  // the normalisation matches what multiplies V.
  uint32_t pk[4];
  float psum = 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float p0 = bf16_round(__builtin_amdgcn_exp2f(sc[h][0] - m_use));
    const float p1 = bf16_round(__builtin_amdgcn_exp2f(sc[h][1] - m_use));
    const float p2 = bf16_round(__builtin_amdgcn_exp2f(sc[h][2] - m_use));
    const float p3 = bf16_round(__builtin_amdgcn_exp2f(sc[h][3] - m_use));
    psum += (p0 + p1) + (p2 + p3);
    pk[2 * h] = pack_bf16x2(p0, p1);
    pk[2 * h + 1] = pack_bf16x2(p2, p3);
  }
  st.l = st.l * alpha + psum;
  st.m = m_new;
  const bf16x8 pb = as_bf16x8(make_uint4(pk[0], pk[1], pk[2], pk[3]));
  // O^T += V^T P^T over this wave's d blocks.  V element q of this lane is
  // key t0 + 8kq + q.  Keys at or past key_end, and keys of an invalid page,
  // may hold anything (even NaN): zero their V so that 0 * V stays 0.
  uint4 vop[8];
  ring_read_v<NE>(base + (R::kKOps + e_lo) * 1024, vop);
  if (!full) {
    const int tb = page_ok ? t0 + 8 * kq : key_end;
    uint32_t vmask[4];
#pragma unroll
    for (int w = 0; w < 4; ++w)
      vmask[w] = (tb + 2 * w < key_end ? 0x0000FFFFu : 0u) |
                 (tb + 2 * w + 1 < key_end ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int u = 0; u < NE; ++u) {
      vop[u].x &= vmask[0];
      vop[u].y &= vmask[1];
      vop[u].z &= vmask[2];
      vop[u].w &= vmask[3];
    }
  }
#pragma unroll
  for (int u = 0; u < NE; ++u) {
    st.o[u] *= alpha;
    st.o[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vop[u]), pb, st.o[u], 0, 0, 0);
  }
}

// Writes a finished row tile for the wave's `ne` d blocks from e_lo: bf16
// output when the piece is the whole segment, otherwise the fp32 partial in
// this workgroup's slot (0: the segment where its share starts, 1: where it
// ends).  (m, l) are identical in every wave of a row tile; the wave that
// owns d block 0 writes them.
template <int D>
__device__ __forceinline__ void write_tile(const AttnParams &p, int g, bool complete, int slot,
                                           const ReqMeta &rq, int rt, int e_lo, int ne,
                                           int lane, const RowState<D> &st) {
  const int kq = lane >> 4, n = lane & 15;
  const int rr = rt * 16 + n;
  if (rr >= p.group * rq.k) return;
  const int lg = __builtin_ctz(p.group);
  const int j = rr >> lg, hh = rr & (p.group - 1);
  if (complete) {
    const size_t row = (size_t)(rq.q0 + j) * p.hq + (size_t)g * p.group + hh;
    const float inv = 1.f / st.l;
    uint16_t *o = p.out + row * D + 16 * e_lo + 4 * kq;
#pragma unroll
    for (int u = 0; u < D / 16; ++u) {
      if (u >= ne) break;
      uint2 w;
      w.x = pack_bf16x2(st.o[u][0] * inv, st.o[u][1] * inv);
      w.y = pack_bf16x2(st.o[u][2] * inv, st.o[u][3] * inv);
      *reinterpret_cast<uint2 *>(o + 16 * u) = w;
    }
  } else {
    const size_t prow = ((size_t)blockIdx.x * 2 + slot) * (p.group * kMaxQlen) + rr;
    float *o = p.part_o + prow * D + 16 * e_lo + 4 * kq;
#pragma unroll
    for (int u = 0; u < D / 16; ++u) {
      if (u >= ne) break;
      *reinterpret_cast<f32x4 *>(o + 16 * u) = st.o[u];
    }
    if (kq == 0 && e_lo == 0) p.part_ml[prow] = make_float2(st.m, st.l);
  }
}

// This workgroup's share of the flattened work: [start, end) in units of
// keys over the segments laid end to end (request-major, then KV head).
struct Share {
  int start, end;
  int i, g, off;  // segment and key offset where `start` falls
};

// Computes the share with one block-wide scan over the requests' segment
// lengths (each thread owns a contiguous run of requests).  Workgroup 0 also
// publishes the per-request prefix and the share size for the combine kernel.
__device__ Share plan_share(const AttnParams &p, int *lds) {
  const int B = p.num_reqs, tid = threadIdx.x;
  const int lane = tid % kWave, wave = tid / kWave;
  const int per = (B + kThreads - 1) / kThreads;
  const int lo = min(B, tid * per), hi = min(B, lo + per);
  int sum = 0;
#pragma unroll 4
  for (int i = lo; i < hi; ++i) sum += segment_len(p, i);
  int incl = sum;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int y = __shfl_up(incl, d, kWave);
    if (lane >= d) incl += y;
  }
  if (lane == kWave - 1) lds[wave] = incl;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    before += w < wave ? lds[w] : 0;
    total += lds[w];
  }
  const int excl = before + incl - sum;  // prefix of this thread's first request
  const int work = total * p.hkv;
  int share = (work + (int)gridDim.x - 1) / (int)gridDim.x;
  share = max(kBlockKeys, round_up_block(share));
  const int start = (int)blockIdx.x * share;
  const int end = min(work, start + share);
  if (blockIdx.x == 0) {
    int acc = excl;
    for (int i = lo; i < hi; ++i) {
      p.plan[i] = acc;
      acc += segment_len(p, i);
    }
    if (tid == 0) {
      p.plan[B] = total;
      p.plan[B + 1] = share;
    }
  }
  // the thread whose requests contain `start` locates it
  if (start < work && excl * p.hkv <= start && start < (excl + sum) * p.hkv) {
    int acc = excl;
    for (int i = lo; i < hi; ++i) {
      const int seg = segment_len(p, i);
      if (start < (acc + seg) * p.hkv) {
        const int rel = start - acc * p.hkv;
        lds[kWaves + 0] = i;
        lds[kWaves + 1] = rel / seg;
        lds[kWaves + 2] = rel % seg;
        break;
      }
      acc += seg;
    }
  }
  __syncthreads();
  Share sh;
  sh.start = start;
  sh.end = end;
  if (start < work) {
    sh.i = __builtin_amdgcn_readfirstlane(lds[kWaves + 0]);
    sh.g = __builtin_amdgcn_readfirstlane(lds[kWaves + 1]);
    sh.off = __builtin_amdgcn_readfirstlane(lds[kWaves + 2]);
  } else {
    sh.i = sh.g = sh.off = 0;
  }
  return sh;
}

// Page id of page k (uniform, k < 128) of the current sub-piece, held one per
// lane in two registers; -1 past the sub-piece.
__device__ __forceinline__ int sub_page(int lo, int hi, int k, int npg) {
  if (k >= npg) return -1;
  return k < kWave ? __builtin_amdgcn_readlane(lo, k) : __builtin_amdgcn_readlane(hi, k - kWave);
}

// One pipeline step: wait for block b, load block b + kStages - 1 into the
// stage block b - 1 used, compute block b.  The ring stages are separate LDS
// arrays and the block loop is unrolled by the stage count, so every ring
// load names a fixed array.
template <int D, int NE>
__device__ __forceinline__ void ring_step(const AttnParams &p, const uint4 (*cur)[kWave],
                                          uint4 (*nxt)[kWave], int g, int b, int nblk, int npg,
                                          int pid_lo, int pid_hi, int wave, int lane,
                                          bool active, int sb, int se, int ctx, int row_limit,
                                          const bf16x8 (&qv)[D / 32], int e_lo,
                                          RowState<D> &st) {
  using R = RingShape<D>;
  // this wave's loads of block b are done once at most the loads of the
  // kStages-2 later blocks are outstanding; the barrier makes every wave's
  // part visible and frees the stage that block b-1 used
  __builtin_amdgcn_s_waitcnt(waitcnt_imm((kStages - 2) * R::kOpsPerWave, 0));
  wg_barrier();
  const int bn = min(b + kStages - 1, nblk - 1);  // clamped: extra loads land unread
  ring_load<D>(p, g, sub_page(pid_lo, pid_hi, 2 * bn, npg),
               sub_page(pid_lo, pid_hi, 2 * bn + 1, npg), nxt, wave, lane);
  if (active) {
    const int c0 = sub_page(pid_lo, pid_hi, 2 * b, npg);
    const int c1 = sub_page(pid_lo, pid_hi, 2 * b + 1, npg);
    const bool ok0 = (unsigned)c0 < (unsigned)p.num_pages;
    const bool ok1 = (unsigned)c1 < (unsigned)p.num_pages;
    const int t0 = sb + b * kBlockKeys;
    const bool full = ok0 && ok1 && t0 + kBlockKeys <= min(ctx, se);
    ring_compute<D, NE>(cur, lane, t0, se, row_limit, full, ok0, ok1, qv, e_lo, p.scale_log2,
                        st);
  }
}

// All blocks of one sub-piece (at most kSubPages pages) through the ring.
template <int D, int NE>
__device__ __forceinline__ void ring_run(const AttnParams &p, uint4 (*r0)[kWave],
                                         uint4 (*r1)[kWave], uint4 (*r2)[kWave],
                                         uint4 (*r3)[kWave], int i, int g, int wave, int lane,
                                         bool active, int sb, int se, int ctx, int row_limit,
                                         const bf16x8 (&qv)[D / 32], int e_lo, RowState<D> &st) {
  static_assert(kStages == 4, "the block loop below is unrolled for four stages");
  const int npg = (se - sb + kPage - 1) / kPage;
  const int nblk = (se - sb + kBlockKeys - 1) / kBlockKeys;
  // this sub-piece's page ids, one per lane in two registers
  const int *pt = p.page_table + (size_t)i * p.max_pages + sb / kPage;
  const int pid_lo = lane < npg ? pt[lane] : -1;
  const int pid_hi = kWave + lane < npg ? pt[kWave + lane] : -1;
  // prologue: the first kStages-1 blocks
  ring_load<D>(p, g, sub_page(pid_lo, pid_hi, 0, npg), sub_page(pid_lo, pid_hi, 1, npg), r0,
               wave, lane);
  {
    const int b1 = min(1, nblk - 1), b2 = min(2, nblk - 1);
    ring_load<D>(p, g, sub_page(pid_lo, pid_hi, 2 * b1, npg),
                 sub_page(pid_lo, pid_hi, 2 * b1 + 1, npg), r1, wave, lane);
    ring_load<D>(p, g, sub_page(pid_lo, pid_hi, 2 * b2, npg),
                 sub_page(pid_lo, pid_hi, 2 * b2 + 1, npg), r2, wave, lane);
  }
  for (int b = 0; b < nblk; b += kStages) {
    ring_step<D, NE>(p, r0, r3, g, b, nblk, npg, pid_lo, pid_hi, wave, lane, active, sb, se,
                     ctx, row_limit, qv, e_lo, st);
    if (b + 1 < nblk)
      ring_step<D, NE>(p, r1, r0, g, b + 1, nblk, npg, pid_lo, pid_hi, wave, lane, active, sb,
                       se, ctx, row_limit, qv, e_lo, st);
    if (b + 2 < nblk)
      ring_step<D, NE>(p, r2, r1, g, b + 2, nblk, npg, pid_lo, pid_hi, wave, lane, active, sb,
                       se, ctx, row_limit, qv, e_lo, st);
    if (b + 3 < nblk)
      ring_step<D, NE>(p, r3, r2, g, b + 3, nblk, npg, pid_lo, pid_hi, wave, lane, active, sb,
                       se, ctx, row_limit, qv, e_lo, st);
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
  wg_barrier();  // the ring is free for the next sub-piece
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_streamk_kernel(AttnParams p) {
  using R = RingShape<D>;
  __shared__ uint4 ring0[R::kOps][kWave];
  __shared__ uint4 ring1[R::kOps][kWave];
  __shared__ uint4 ring2[R::kOps][kWave];
  __shared__ uint4 ring3[R::kOps][kWave];
  __shared__ int lds_plan[kWaves + 4];

  const Share sh = plan_share(p, lds_plan);
  if (sh.start >= sh.end) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int kq = lane >> 4, n = lane & 15;

  int i = sh.i, g = sh.g, off = sh.off, pos = sh.start, piece = 0;
  while (pos < sh.end && i < p.num_reqs) {
    const ReqMeta rq = load_req(p, i);
    if (rq.seg == 0) {  // sentinel or bad metadata: no keys in the plan
      ++i;
      continue;
    }
    const int take = min(rq.seg - off, sh.end - pos);
    const int key_begin = off, key_end = min(rq.len, off + take);
    const bool complete = off == 0 && take == rq.seg;
    const int slot = piece == 0 ? 0 : 1;

    // Wave roles.  Every wave computes every block of the piece:
    //  1 row tile:  all four waves on it, each with a quarter of the dims;
    //  2 row tiles: two waves per tile, each with half of the dims;
    //  3+ tiles:    one tile per wave, all dims (passes of four tiles).
    const int rows = p.group * rq.k;
    const int nt = (rows + 15) / 16;
    const int nds = nt == 1 ? 4 : (nt == 2 ? 2 : 1);
    const int npass = (nt + kWaves - 1) / kWaves;
    const int ne = (D / 16) / nds;
    for (int pass = 0; pass < npass; ++pass) {
      const int rt = nds > 1 ? wave % nt : wave + kWaves * pass;
      const int ds = nds > 1 ? wave / nt : 0;
      const bool active = rt < nt;
      const int e_lo = ds * ne;
      const int rr = rt * 16 + n;
      const bool valid_row = active && rr < rows;
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
      RowState<D> st;
      st.m = -INFINITY;
      st.l = 0.f;
#pragma unroll
      for (int e = 0; e < D / 16; ++e) st.o[e] = f32x4{0.f, 0.f, 0.f, 0.f};

      for (int sb = key_begin; sb < key_end; sb += kSubPages * kPage) {
        const int se = min(key_end, sb + kSubPages * kPage);
        if (ne == D / 16)
          ring_run<D, D / 16>(p, ring0, ring1, ring2, ring3, i, g, wave, lane, active, sb, se,
                              rq.ctx, row_limit, qv, e_lo, st);
        else if (ne == D / 32)
          ring_run<D, D / 32>(p, ring0, ring1, ring2, ring3, i, g, wave, lane, active, sb, se,
                              rq.ctx, row_limit, qv, e_lo, st);
        else
          ring_run<D, D / 64>(p, ring0, ring1, ring2, ring3, i, g, wave, lane, active, sb, se,
                              rq.ctx, row_limit, qv, e_lo, st);
      }
      if (active) {
        // the lane holds a partial row sum over its own keys; complete it
        st.l += shfl_xor_f(st.l, 16);
        st.l += shfl_xor_f(st.l, 32);
        write_tile<D>(p, g, complete, slot, rq, rt, e_lo, ne, lane, st);
      }
    }

    pos += take;
    off += take;
    ++piece;
    if (off == rq.seg) {
      off = 0;
      if (++g == p.hkv) {
        g = 0;
        ++i;
      }
    }
  }
}

// Merges the partials of segments that straddle share boundaries (in
// workgroup order, so the result is deterministic) and zeroes the tail rows.
// Workgroup (x, g, i) owns 256/(D/4) live rows of request i and KV head g;
// each thread owns 4 output dims of one row and issues the loads of up to 8
// partials at a time.  Workgroups with z == B zero the tail rows instead.
template <int D>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(AttnParams p) {
  constexpr int kLanesPerRow = D / 4;
  constexpr int kRows = kThreads / kLanesPerRow;
  const int g = blockIdx.y, i = blockIdx.z;
  const int G = p.group;
  if (i == p.num_reqs) {
    const int live = min(max(p.cu[p.num_reqs], 0), p.cap);
    const int per_row = G * (D / 8);
    const int total = (p.cap - live) * per_row;
    for (int idx = blockIdx.x * kThreads + threadIdx.x; idx < total;
         idx += gridDim.x * kThreads) {
      const int r = live + idx / per_row, rem = idx % per_row;
      const int hh = rem / (D / 8), d8 = rem % (D / 8);
      uint16_t *o = p.out + ((size_t)r * p.hq + (size_t)g * G + hh) * D + 8 * d8;
      *reinterpret_cast<uint4 *>(o) = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  const int prefix = p.plan[i];
  const int seg = p.plan[i + 1] - prefix;  // p.plan[B] is the total
  if (seg <= 0) return;
  const int share = p.plan[p.num_reqs + 1];
  const int start = prefix * p.hkv + g * seg;
  const int b0 = start / share, b1 = (start + seg - 1) / share;
  if (b0 == b1) return;  // one workgroup held the whole segment
  const ReqMeta rq = load_req(p, i);
  const int rr = blockIdx.x * kRows + threadIdx.x / kLanesPerRow;
  if (rr >= G * rq.k) return;
  const int d4 = threadIdx.x % kLanesPerRow;
  const int lg = __builtin_ctz(G);
  const int j = rr >> lg, hh = rr & (G - 1);
  const size_t row = (size_t)(rq.q0 + j) * p.hq + (size_t)g * G + hh;
  const int n_parts = b1 - b0 + 1;
  // partial of workgroup b0 + u: slot 0 if its share starts inside this
  // segment, else slot 1 (the segment is where its share ends)
  auto prow = [&](int u) -> size_t {
    const int b = b0 + u;
    const int slot = b * share >= start ? 0 : 1;
    return ((size_t)b * 2 + slot) * (G * kMaxQlen) + rr;
  };

  float mx = -INFINITY;
  for (int u0 = 0; u0 < n_parts; u0 += 8) {
    float m8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      m8[u] = u0 + u < n_parts ? p.part_ml[prow(u0 + u)].x : -INFINITY;
#pragma unroll
    for (int u = 0; u < 8; ++u) mx = fmaxf(mx, m8[u]);
  }
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  for (int u0 = 0; u0 < n_parts; u0 += 8) {
    float2 l8[8];
    f32x4 o8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool in = u0 + u < n_parts;
      const size_t pr = prow(u0 + u);
      l8[u] = in ? p.part_ml[pr] : make_float2(-INFINITY, 0.f);
      o8[u] = in ? *reinterpret_cast<const f32x4 *>(p.part_o + pr * D + 4 * d4)
                 : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float w = exp2f(l8[u].x - mx);
      den += w * l8[u].y;
      acc += w * o8[u];
    }
  }
  const float inv = 1.f / den;
  uint2 w2;
  w2.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  w2.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<uint2 *>(p.out + row * D + 4 * d4) = w2;
}

// Workgroups the GPU holds at once for the stream-K kernel (cached per
// device and head dim; a host query, so it is safe during graph capture).
int resident_workgroups(int head_dim) {
  static int cache[64][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int &slot = cache[dev][head_dim == 128 ? 1 : 0];
  if (slot > 0) return slot;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const hipError_t e =
      head_dim == 128
          ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_streamk_kernel<128>, kThreads, 0)
          : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_streamk_kernel<64>, kThreads, 0);
  if (e != hipSuccess || cus <= 0 || per_cu <= 0) return 0;
  slot = cus * per_cu;
  return slot;
}

}  // namespace

// Upper bound of the persistent grid, known without a device: at most 1024
// workgroups (a 256-CU MI355X holds 768 of this kernel at once) and never
// more than the 32-key blocks the largest batch could hold.  The workspace
// is sized for it.
int32_t attn_grid_cap(const dsv_attn_dims &d) {
  constexpr long long kMaxGrid = 1024;
  const long long blocks = (long long)d.num_reqs * d.num_kv_heads *
                           ((d.max_kv_len + kBlockKeys - 1) / kBlockKeys);
  return (int32_t)(blocks < kMaxGrid ? blocks : kMaxGrid);
}

// Launch grid: the workgroups the current device holds at once, capped.
int32_t attn_grid(const dsv_attn_dims &d) {
  const int r = resident_workgroups(d.head_dim);
  if (r <= 0) return 0;
  const int32_t cap = attn_grid_cap(d);
  return r < cap ? r : cap;
}

AttnWorkspace attn_workspace_layout(const dsv_attn_dims &d) {
  AttnWorkspace w;
  const size_t grid = (size_t)attn_grid_cap(d);
  const size_t rows = grid * 2 * (size_t)(d.num_q_heads / d.num_kv_heads) * kMaxQlen;
  w.grid_cap = (int32_t)grid;
  w.plan_off = 0;
  w.part_ml_off = align_up((size_t)(d.num_reqs + 2) * sizeof(int32_t), 256);
  w.part_o_off = align_up(w.part_ml_off + rows * sizeof(float2), 256);
  w.total = align_up(w.part_o_off + rows * d.head_dim * sizeof(float), 256);
  return w;
}

hipError_t launch_verify_attn(const AttnParams &p, int head_dim, hipStream_t s) {
  // rows of one request and KV head: G * k_i <= G * 16
  const int comb_rows = head_dim == 128 ? kThreads / 32 : kThreads / 16;
  const dim3 grid_comb((p.group * kMaxQlen + comb_rows - 1) / comb_rows, p.hkv,
                       p.num_reqs + 1);
  timing_mark(kTimeAttnSplit, false, s);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_streamk_kernel<128>, dim3(p.num_wg), dim3(kThreads), 0, s, p);
  else
    hipLaunchKernelGGL(attn_streamk_kernel<64>, dim3(p.num_wg), dim3(kThreads), 0, s, p);
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
