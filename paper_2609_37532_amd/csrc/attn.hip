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
//    ceil32(ctx_i + k_i) keys; the segments are laid end to end, each
//    after a lead-in of six blocks that stands for the cost of starting a
//    piece on it, and a persistent grid, sized to the workgroups the GPU
//    holds at once, gives every workgroup one contiguous share of that
//    space (streaming plus piece starts), equal up to a small skew by grid
//    index parity for the XCDs' unequal streaming rates.  A workgroup walks the
//    segments its share touches; a segment it covers whole is written as
//    bf16 directly, a segment cut at a share boundary leaves an fp32 partial
//    (O, m, l) that the combine kernel merges in workgroup order.  Ragged
//    contexts cost no idle workgroups, and there are at most two partials
//    per workgroup.  Results depend only on the request's own data and the
//    batch's total work (the share size), and merge in a fixed order, so
//    they are deterministic.  Small batches, whose even share would fall
//    below eight blocks, instead cut every segment into equal block-aligned
//    pieces, one per workgroup, so that no workgroup straddles two segments.
//  * K/V stream through an LDS ring of three 32-key blocks.  Each wave
//    loads one 4 KiB tile per block (one page's K or V) into registers
//    three blocks ahead, as four contiguous 1 KiB loads from a scalar page
//    address, and writes it to the ring when its block comes up; on gfx950
//    this sustains more bandwidth than LDS-direct loads.  Page ids are
//    staged in LDS per piece.
//  * Transposed scores: S^T = K Q^T and O^T = V^T P^T with
//    v_mfma_f32_16x16x32_bf16.  The score tile comes out with one query row
//    per lane column, which is exactly the B-operand layout the PV product
//    needs, so P never crosses lanes; the row max and the row sum each need
//    two row-swap permutes.  Each weight enters PV as a hi + lo pair of bf16
//    values (two MFMAs per output tile), so the weights carry about 2^-17
//    of their value and the output's own bf16 rounding dominates the error.
//  * Lazy rescaling: the running maximum only moves (and the accumulators
//    are only rescaled) when a block's maximum exceeds it by more than a
//    factor 2^8, which keeps the weights below 2^8.  It is kept an integer,
//    so rescales and merge weights are exact powers of two.
//  * Waves of a workgroup split the dims when a request has one or two row
//    tiles; with three or more row tiles each wave owns tiles.
//  * The workgroup placed second on a CU runs at raised wave priority over
//    most of its share, so that both workgroups of a CU finish together.
#include "dsv_internal.h"

#include <math.h>

namespace dsv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
// Combine kernel: 1024-thread workgroups (32 rows at D = 128) need a quarter
// of the workgroups that 256 threads do, most of which exit at once; measured
// 0.6 us faster at B=32 with contexts up to 8K (Qwen3-8B attention shape).
constexpr int kCombThreads = 1024;
constexpr int kBlockKeys = kAttnBlockKeys;  // keys per inner step (two pages)
// Smallest stream-K share: with little work (short contexts, few requests)
// eight blocks per workgroup beat spreading it over every resident
// workgroup -- fewer cut segments, so less partial traffic and combine work,
// and a longer pipeline per workgroup.
constexpr int kMinShare = 8 * kBlockKeys;
// Stream-K lead-in: every segment with keys counts kLeadKeys more in the
// linear work space than it holds, the cost of starting a piece on it
// (metadata, page ids, query rows, the ring's first blocks), so that equal
// shares are equal in streaming plus piece starts.  A multiple of the block;
// six blocks measured best across shapes (two to eight were compared).
constexpr int kLeadKeys = kAttnLeadKeys;
// Wave priority.  The persistent grid holds two workgroups per CU, and the
// one the dispatcher places second (grid index >= number of CUs) loses
// instruction arbitration to the older first one: with equal shares it
// finished several microseconds later, and the CU's last stretch ran on one
// workgroup.  Its waves therefore run at raised priority until kBoostPct
// percent of its share is done, then at the default.  Priority changes no
// arithmetic.  Drop points of 50, 65, 80 and 90 percent and the whole share
// were compared; 65 gained the most over shapes.
constexpr int kBoostPct = 65;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

// Two bf16 -> one uint32 (low half first), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
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
// One 32-key block (two pages) in LDS: the K tiles of both pages, then their
// V tiles, each tile as D/32 chunks of 1 KiB.  Wave w stages page w & 1's K
// (waves 0-1) or V (waves 2-3) tile of every block.  Lane l writes the 16
// bytes at offset 16*l of each chunk and loads a swizzled 16-byte unit of
// it (each aligned group of four lanes still reads one aligned 64-byte
// piece), chosen so that the MFMA operand reads are free of LDS bank
// conflicts for any grouping of 8, 16 or 32 lanes per LDS cycle (k_unit /
// v_unit below).
template <int D>
struct Ring {
  static constexpr int kChunks = D / 32;               // 1 KiB chunks per tile
  static constexpr int kKRegion = 2 * kChunks * 1024;  // K tiles of both pages
  static constexpr int kStage = 2 * kKRegion;          // 16 KiB at D = 128
  static constexpr int kKOps = 2 * kChunks;            // K operand tiles per block
};
// Ring stages = blocks in flight in registers.  Four (16 more VGPRs, 64 KiB
// of ring) measured 1-3% slower than three at every shape.
constexpr int kStages = 3;
constexpr int kSubPages = 512;  // page ids staged in LDS at a time (8192 keys)

// The wave's share of one block: one page's K or V tile (D/32 chunks of
// 1 KiB), loaded into registers (lane l holds the swizzled unit it will
// write at offset 16*l of each chunk) and later written to its ring stage.
template <int D>
struct StageRegs {
  u32x4 x[D / 32];
};

template <int D>
__device__ __forceinline__ void stage_load(const char *tile, uint32_t voff, StageRegs<D> &r) {
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
    r.x[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(tile + voff + 1024 * c));
}

template <int D>
__device__ __forceinline__ void stage_store(char *dst, int lane, const StageRegs<D> &r) {
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
    *reinterpret_cast<u32x4 *>(dst + 1024 * c + 16 * lane) = r.x[c];
}

// Key order inside a block.  Row m of score half hh holds key
// 8*(m/4) + 4*hh + m%4, so after S^T = K Q^T the lane with k-group kq holds
// keys 8*kq + [0..7] of its query row: exactly the order the PV product
// contracts over, and V's operand for that lane is 8 consecutive keys of one
// dim, one 16-byte unit of the d-major V tile.
__device__ __forceinline__ int score_key(int hh, int m) { return 8 * (m >> 2) + 4 * hh + (m & 3); }

// Swizzles.  K chunk of page p: global unit u (d-chunk u/16, slot u%16)
// sits at LDS unit k_unit(u, p) (an involution).  V chunk: global unit
// u = 2*dim + half sits at LDS unit v_unit(u); v_unit_inv is its inverse.
__device__ __forceinline__ int k_unit(int u, int p) { return u ^ (4 * (p ^ ((u >> 3) & 1))); }
__device__ __forceinline__ int v_sel(int k) { return ((k >> 1) ^ (k >> 2)) & 1; }
__device__ __forceinline__ int v_unit(int u) {
  const int k = u >> 2, j = (u >> 1) & 1, b = u & 1;
  return 4 * k + 2 * (b ^ v_sel(k)) + j;
}
__device__ __forceinline__ int v_unit_inv(int l) {
  const int k = l >> 2, j = l & 1, b = ((l >> 1) & 1) ^ v_sel(k);
  return 4 * k + 2 * j + b;
}

// Per-lane LDS byte offsets (within a stage) of the MFMA operands.
struct RingLane {
  uint32_t k0, k1;  // K operand, score half 0 / 1, chunk 0 (chunk c at +1024c)
  uint32_t v;       // V operand of d block 0 (d block e at +512e)
};

template <int D>
__device__ __forceinline__ RingLane ring_lane(int lane) {
  using R = Ring<D>;
  const int kgrp = lane >> 4, m = lane & 15;
  RingLane r;
  {
    const int key0 = score_key(0, m), key1 = score_key(1, m);
    const int p0 = key0 >> 4, p1 = key1 >> 4;
    r.k0 = (uint32_t)(p0 * R::kChunks * 1024 + 16 * k_unit(kgrp * 16 + (key0 & 15), p0));
    r.k1 = (uint32_t)(p1 * R::kChunks * 1024 + 16 * k_unit(kgrp * 16 + (key1 & 15), p1));
  }
  {
    // dim m of d block 0, keys 8*(kgrp&1) .. +7 of page kgrp>>1
    const int pv = kgrp >> 1;
    r.v = (uint32_t)(R::kKRegion + pv * R::kChunks * 1024 + 16 * v_unit(2 * m + (kgrp & 1)));
  }
  return r;
}

// Maximum / sum over the four lanes that hold one query row (lanes n, n+16,
// n+32, n+48), with the gfx950 row-swap permutes.
__device__ __forceinline__ float row_max4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Sum over the same four lanes.  Each swap hands every lane the pair in the
// same order, so the four lanes end with bitwise equal sums.
__device__ __forceinline__ float row_sum4(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// The running maximum is only raised when a block's maximum exceeds it by
// more than this (base-2 units): weights then stay below 2^8, and the
// accumulators are rescaled only on such a jump instead of every block.
// The maximum is kept an integer (the block maximum rounded up), so every
// rescale factor and every merge weight of the combine is an exact power of
// two: where a segment is cut, or which rows share its tile, moves a row's
// weights and sums by powers of two only, and its result changes only
// through fp32 summation order.
constexpr float kRescaleSlack = 8.f;

// Online-softmax state of one lane: one query row (lane & 15); `l` holds
// the row sum of the weights (the same value in the row's four lanes);
// for each of the wave's d blocks u (dims 16*(e_lo+u) + 4*(lane>>4) +
// [0..3]), the 4 accumulated outputs.
template <int D>
struct RowState {
  float m;
  float l;
  f32x4 o[D / 16];
};

// One 32-key block from ring stage byte offset `so`: scores for the wave's
// row tile, online softmax, and the PV product for the wave's NE d blocks
// starting at e_lo (`vb` already points at e_lo).  `full` (uniform) says every
// key of the block is visible to every live row, so no masking is needed.
template <int D, int NE>
__device__ __forceinline__ void ring_compute(const char *ring, uint32_t so, const RingLane &rl,
                                             uint32_t vb, int lane, int t0, int key_end,
                                             int row_limit, bool full,
                                             const bf16x8 (&qv)[D / 32], float scale_log2,
                                             RowState<D> &st) {
  using R = Ring<D>;
  const int kq = lane >> 4;
  uint4 kop[R::kKOps];
#pragma unroll
  for (int c = 0; c < R::kChunks; ++c) {
    kop[c] = *reinterpret_cast<const uint4 *>(ring + so + rl.k0 + 1024 * c);
    kop[R::kChunks + c] = *reinterpret_cast<const uint4 *>(ring + so + rl.k1 + 1024 * c);
  }
  uint4 vop[NE];
#pragma unroll
  for (int u = 0; u < NE; ++u) vop[u] = *reinterpret_cast<const uint4 *>(ring + so + vb + 512 * u);
  f32x4 s[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    s[h] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
      s[h] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kop[h * (D / 32) + c]), qv[c],
                                                     s[h], 0, 0, 0);
  }
  // element (h, q) of this lane is key t0 + 8kq + 4h + q; raw scores (the
  // scale is positive and applied inside the exponent)
  float sc[2][4];
  if (full) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q) sc[h][q] = s[h][q];
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = t0 + 8 * kq + 4 * h + q;
        const bool vis = t <= row_limit && t < key_end;
        sc[h][q] = vis ? s[h][q] : -INFINITY;
      }
  }
  float bmax = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                     fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
  bmax = row_max4(bmax) * scale_log2;
  if (__builtin_amdgcn_ballot_w64(bmax > st.m + kRescaleSlack) != 0) {
    const float m_new = fmaxf(st.m, ceilf(bmax));
    // 0 on a row's first visible block, 1 for a row that still sees nothing
    const float alpha = __builtin_amdgcn_exp2f(st.m - (m_new == -INFINITY ? 0.f : m_new));
    st.l *= alpha;
#pragma unroll
    for (int u = 0; u < NE; ++u) st.o[u] *= alpha;
    st.m = m_new;
  }
  const float neg_m = st.m == -INFINITY ? 0.f : -st.m;
  // P enters the bf16 PV product as a pair: hi = P rounded to bf16 and
  // lo = the remainder rounded to bf16, so hi + lo carries P to about 2^-17
  // of its value and the weights add no error next to the output's own bf16
  // rounding.  The row sum adds the fp32 weights themselves: the lane's
  // eight, then across the row's four lanes.
  uint32_t pk[4], pl[4];
  float psum = 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    float pw[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      pw[q] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[h][q], scale_log2, neg_m));
    psum += (pw[0] + pw[1]) + (pw[2] + pw[3]);
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      const uint32_t hi = pack_bf16x2(pw[2 * w], pw[2 * w + 1]);
      pk[2 * h + w] = hi;
      pl[2 * h + w] = pack_bf16x2(pw[2 * w] - __uint_as_float(hi << 16),
                                  pw[2 * w + 1] - __uint_as_float(hi & 0xFFFF0000u));
    }
  }
  const bf16x8 pb = as_bf16x8(make_uint4(pk[0], pk[1], pk[2], pk[3]));
  const bf16x8 pbl = as_bf16x8(make_uint4(pl[0], pl[1], pl[2], pl[3]));
  // V element q of this lane is key t0 + 8kq + q.  Keys at or past key_end
  // may hold anything (even NaN): zero their V so that 0 * V stays 0.
  if (!full) {
    const int tb = t0 + 8 * kq;
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
  for (int u = 0; u < NE; ++u)
    st.o[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vop[u]), pb, st.o[u], 0, 0, 0);
#pragma unroll
  for (int u = 0; u < NE; ++u)
    st.o[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vop[u]), pbl, st.o[u], 0, 0, 0);
  st.l += row_sum4(psum);
}

// Writes a finished row tile for the wave's `ne` d blocks from e_lo: bf16
// output when the piece is the whole segment, otherwise the fp32 partial in
// this workgroup's slot (0: the segment where its share starts, 1: where it
// ends).  (m, l) are identical in every wave of a row tile; the wave that
// owns d block 0 writes them.
template <int D>
__device__ __forceinline__ void write_tile(const AttnParams &p, int g, bool complete, int slot,
                                           const ReqMeta &rq, int rt, int e_lo, int ne,
                                           int lane, float l, const RowState<D> &st) {
  const int kq = lane >> 4, n = lane & 15;
  const int rr = rt * 16 + n;
  if (rr >= p.group * rq.k) return;
  const int lg = __builtin_ctz(p.group);
  const int j = rr >> lg, hh = rr & (p.group - 1);
  if (complete) {
    const size_t row = (size_t)(rq.q0 + j) * p.hq + (size_t)g * p.group + hh;
    const float inv = 1.f / l;
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
    if (kq == 0 && e_lo == 0) p.part_ml[prow] = make_float2(st.m, l);
  }
}

// This workgroup's share of the flattened work: [start, end) in units of
// keys over the segments laid end to end (request-major, then KV head).
struct Share {
  int start, end;
  int i, g, off;  // segment and virtual offset where `start` falls
  int lead;       // keys of lead-in per segment: kLeadKeys (stream-K) or 0
  ReqMeta first;  // request i's metadata, as read by the plan
};

// Small batches.  When the even share falls to the minimum, each segment is
// instead cut into pieces of at most `cap` keys, as equal as whole blocks
// allow, one piece per workgroup: no workgroup then pays for a second piece
// (its metadata, page ids and pipeline refill), which at this size is a
// large part of the kernel.  The cap is the smallest of kPieceCaps blocks
// that leaves at most one piece per CU -- a second workgroup on a CU shares
// its MFMA and LDS with the first and finishes last -- else the smallest,
// if the pieces fit the grid.  Piece q of n of a `seg`-key segment starts at
// piece_begin(seg, n, q).
constexpr int kNumPieceCaps = 5;
__device__ __forceinline__ int piece_cap(int c) { return (8 + c) * kBlockKeys; }  // 8..12 blocks
__device__ __forceinline__ int seg_pieces(int seg, int cap) { return (seg + cap - 1) / cap; }
__device__ __forceinline__ int piece_begin(int seg, int n, int q) {
  return (int)((long long)(seg / kBlockKeys) * q / n) * kBlockKeys;
}

// Stream-K shares alternate in size with the workgroup's grid index.  The
// dispatcher places workgroup b on XCD b mod 8, and with equal shares the
// workgroups on the odd XCDs finished 6-10 us after those on the even ones
// in every clocked launch of the Qwen3-8B shape at B=32, contexts up to 8K,
// while the shader clocks of all eight XCDs agreed within 2%.  Even
// workgroups therefore take kSkewPct percent more than the mean share and
// odd ones as much less (whole blocks).
constexpr int kSkewPct = 6;
__device__ __forceinline__ int share_skew(int share) {
  return (int)((long long)share * kSkewPct / 100) / kBlockKeys * kBlockKeys;
}
// First virtual key of workgroup b's share.
__device__ __forceinline__ int share_begin(int b, int share, int skew) {
  return b * share + (b & 1) * skew;
}
// The workgroup whose share holds virtual key pos.
__device__ __forceinline__ int share_owner(int pos, int share, int skew) {
  const int pair = pos / (2 * share);
  return 2 * pair + (pos - pair * 2 * share >= share + skew ? 1 : 0);
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP row shifts and
// row broadcasts (lanes without a source add 0): six VALU steps, where a
// shuffle-based scan would take six LDS permutes.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int dpp_src(int v) {
  return __builtin_amdgcn_update_dpp(0, v, kCtrl, kRowMask, 0xf, false);
}
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += dpp_src<0x111, 0xf>(v);  // row_shr:1
  v += dpp_src<0x112, 0xf>(v);  // row_shr:2
  v += dpp_src<0x114, 0xf>(v);  // row_shr:4
  v += dpp_src<0x118, 0xf>(v);  // row_shr:8
  v += dpp_src<0x142, 0xa>(v);  // row_bcast:15
  v += dpp_src<0x143, 0xc>(v);  // row_bcast:31
  return v;
}

// Block-wide exclusive scan of one value per thread: the wave scan, then the
// wave totals through LDS (`tot` receives the block total).
__device__ __forceinline__ int block_excl_scan(int v, int *lds_tot, int &tot) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int incl = wave_incl_scan(v);
  if (lane == kWave - 1) lds_tot[wave] = incl;
  __syncthreads();
  int before = 0;
  tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    before += w < wave ? lds_tot[w] : 0;
    tot += lds_tot[w];
  }
  return before + incl - v;
}

// Computes the share with block-wide scans over the requests' segment
// lengths (each thread owns a contiguous run of requests): a stream-K share
// of the flattened work, or, for small batches, one piece of one segment.
// Workgroup 0 also publishes the per-request prefixes and the plan for the
// combine kernel.  LDS use: lds[0..2*kWaves) scan totals, then the located
// share.
__device__ Share plan_share(const AttnParams &p, int *lds) {
  const int B = p.num_reqs, tid = threadIdx.x;
  const int per = (B + kThreads - 1) / kThreads;
  const int lo = min(B, tid * per), hi = min(B, lo + per);
  int sum = 0;
  // with one request per thread (B <= 256) its metadata stays in registers
  // for the locate step below
  int q0 = 0, q1 = 0, cx = 0;
  if (per == 1) {
    if (lo < hi) {
      q0 = p.cu[lo];
      q1 = p.cu[lo + 1];
      cx = p.ctx[lo];
      sum = segment_of(p, q0, q1, cx);
    }
  } else {
#pragma unroll 4
    for (int i = lo; i < hi; ++i) sum += segment_len(p, i);
  }
  int total;
  const int excl = block_excl_scan(sum, lds, total);  // keys before my requests
  int *loc = lds + 2 * kWaves;  // located share: i, g, off, q0, q1, ctx, start, end
  const int work = total * p.hkv;
  int share = (work + (int)gridDim.x - 1) / (int)gridDim.x;
  share = max(kMinShare, round_up_block(share));
  // Small batch: the even share is at the minimum.  Count the segment pieces
  // under every candidate cap (block totals only: one wave sum per cap, one
  // barrier) and pick the cap; every workgroup computes the same choice.
  int cap = 0;
  if (share == kMinShare) {
    int cnt[kNumPieceCaps];
#pragma unroll
    for (int c = 0; c < kNumPieceCaps; ++c) cnt[c] = 0;
    for (int i = lo; i < hi; ++i) {
      const int seg = per == 1 ? sum : segment_len(p, i);
#pragma unroll
      for (int c = 0; c < kNumPieceCaps; ++c) cnt[c] += seg_pieces(seg, piece_cap(c));
    }
    int *red = loc + 8;  // [kNumPieceCaps][kWaves]
    const int lane = tid % kWave, wave = tid / kWave;
#pragma unroll
    for (int c = 0; c < kNumPieceCaps; ++c) {
      const int v = wave_incl_scan(cnt[c]);
      if (lane == kWave - 1) red[c * kWaves + wave] = v;
    }
    __syncthreads();
    // every piece needs a workgroup of the grid
    const int one_per_cu = min(p.num_cu, (int)gridDim.x);
    for (int c = kNumPieceCaps - 1; c >= -1; --c) {
      // the smallest cap with at most one piece per CU; failing that the
      // smallest cap if its pieces fit the grid
      const int cc = c < 0 ? 0 : c;
      int t = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) t += red[cc * kWaves + w];
      if (c >= 0 ? t * p.hkv <= one_per_cu : t * p.hkv <= (int)gridDim.x && cap == 0)
        cap = piece_cap(cc);
    }
  }
  const bool seg_mode = cap > 0;
  int npc = 0;
  if (seg_mode) {
    if (per == 1) {
      npc = seg_pieces(sum, cap);
    } else {
      for (int i = lo; i < hi; ++i) npc += seg_pieces(segment_len(p, i), cap);
    }
  }
  // Stream-K works in the virtual space where each segment with keys is
  // lead keys longer (its lead-in first); the small-batch plan in keys.
  const int lead = seg_mode ? 0 : kLeadKeys;
  int total_pc = 0, total_v = total, excl_pc = 0, excl_v = excl, sum_v = sum;
  if (seg_mode) {
    excl_pc = block_excl_scan(npc, lds + kWaves, total_pc);
  } else {
    int nnz = 0;  // this thread's segments with keys
    if (per == 1) {
      nnz = sum > 0 ? 1 : 0;
    } else {
      for (int i = lo; i < hi; ++i) nnz += segment_len(p, i) > 0 ? 1 : 0;
    }
    sum_v = sum + lead * nnz;
    excl_v = block_excl_scan(sum_v, lds + kWaves, total_v);
    const int work_v = total_v * p.hkv;
    share = (work_v + (int)gridDim.x - 1) / (int)gridDim.x;
    share = max(kMinShare, round_up_block(share));
  }
  const int work_s = total_v * p.hkv;  // the plan's linear space (= work when seg_mode)
  if (blockIdx.x == 0) {
    int acc = excl_v, acc_pc = excl_pc;
    for (int i = lo; i < hi; ++i) {
      const int seg = segment_len(p, i);
      p.plan[i] = acc;
      p.plan[B + 2 + i] = acc_pc;
      acc += seg > 0 ? seg + lead : 0;
      if (seg_mode) acc_pc += seg_pieces(seg, cap);
    }
    if (tid == 0) {
      p.plan[B] = total_v;
      p.plan[B + 1] = seg_mode ? -cap : share;  // negative: the small-batch cap
      p.plan[2 * B + 2] = total_pc;
    }
  }
  const int b = (int)blockIdx.x;
  int start = work_s, end = work_s;
  if (!seg_mode) {
    const int skew = share_skew(share);
    start = min(work_s, share_begin(b, share, skew));
    end = min(work_s, share_begin(b + 1, share, skew));
  }
  // the thread whose requests contain this workgroup's share locates it and
  // publishes the request's metadata, so the first piece needs no second
  // read of it
  const bool mine = seg_mode ? (b < total_pc * p.hkv && excl_pc * p.hkv <= b &&
                                b < (excl_pc + npc) * p.hkv)
                             : (start < work_s && excl_v * p.hkv <= start &&
                                start < (excl_v + sum_v) * p.hkv);
  if (mine) {
    int acc = excl_v, acc_pc = excl_pc;
    for (int i = lo; i < hi; ++i) {
      if (per != 1) {
        q0 = p.cu[i];
        q1 = p.cu[i + 1];
        cx = p.ctx[i];
      }
      const int seg = segment_of(p, q0, q1, cx);
      const int segv = seg > 0 ? seg + lead : 0;  // seg when seg_mode
      const int n = seg_mode ? seg_pieces(seg, cap) : 0;
      int g = -1, off = 0, s0 = 0, s1 = 0;
      if (seg_mode) {
        if (b < (acc_pc + n) * p.hkv) {
          const int rel = b - acc_pc * p.hkv;
          g = rel / n;
          const int q = rel % n;
          off = piece_begin(seg, n, q);
          s0 = acc * p.hkv + g * seg + off;
          s1 = s0 + piece_begin(seg, n, q + 1) - off;
        }
      } else if (start < (acc + segv) * p.hkv) {
        const int rel = start - acc * p.hkv;
        g = rel / segv;
        off = rel % segv;
        s0 = start;
        s1 = end;
      }
      if (g >= 0) {
        loc[0] = i;
        loc[1] = g;
        loc[2] = off;
        loc[3] = q0;
        loc[4] = q1;
        loc[5] = cx;
        loc[6] = s0;
        loc[7] = s1;
        break;
      }
      acc += segv;
      acc_pc += n;
    }
  }
  __syncthreads();
  Share sh;
  sh.lead = lead;
  const bool has = seg_mode ? b < total_pc * p.hkv : start < work_s;
  if (has) {
    sh.start = __builtin_amdgcn_readfirstlane(loc[6]);
    sh.end = __builtin_amdgcn_readfirstlane(loc[7]);
    sh.i = __builtin_amdgcn_readfirstlane(loc[0]);
    sh.g = __builtin_amdgcn_readfirstlane(loc[1]);
    sh.off = __builtin_amdgcn_readfirstlane(loc[2]);
    const int f0 = __builtin_amdgcn_readfirstlane(loc[3]);
    const int f1 = __builtin_amdgcn_readfirstlane(loc[4]);
    sh.first.q0 = f0;
    sh.first.ctx = __builtin_amdgcn_readfirstlane(loc[5]);
    sh.first.k = f1 - f0;
    sh.first.len = sh.first.ctx + sh.first.k;
    sh.first.seg = segment_of(p, f0, f1, sh.first.ctx);
  } else {
    sh.start = sh.end = work_s;
    sh.i = sh.g = sh.off = 0;
    sh.first = ReqMeta{0, 0, 0, 0, 0};
  }
  return sh;
}

// Everything a wave needs to run the ring over one sub-piece.
template <int D>
struct RingCtx {
  const char *ring;      // LDS ring base
  const int *pg;         // LDS page ids of the sub-piece (sanitised)
  const char *kvw;       // this wave's tile of page 0: kv + (kind*Hkv + g) tiles
  size_t page_bytes;     // bytes per page (2 * Hkv tiles)
  uint32_t dst0;         // byte offset of this wave's tile region in a stage
  uint32_t voff;         // this lane's swizzled global offset inside a chunk
  int pp;                // page parity this wave loads
  RingLane rl;
  uint32_t vb;           // V operand offset of the wave's first d block
  int nblk;              // blocks in the sub-piece
  int sb, se, ctx, row_limit;
  int prio_end_b;        // block at which the wave priority returns to the default
  bool active;
};

// Address of this wave's tile of block b (clamped: past the end it reloads
// the last block, which is never read).
template <int D>
__device__ __forceinline__ const char *tile_of(const RingCtx<D> &c, int b) {
  const int bb = min(b, c.nblk - 1);
  const int pid = __builtin_amdgcn_readfirstlane(c.pg[2 * bb + c.pp]);
  return c.kvw + (size_t)pid * c.page_bytes;
}

// One pipeline step with block b in compile-time stage ST: write the wave's
// tile of block b (in registers since three steps ago) to the stage, start
// loading block b + kStages into those registers, and after the barrier
// compute block b.  The stage was last read at step b - kStages, which every
// wave finished before the barrier of step b - kStages + 1.
template <int D, int NE, int ST>
__device__ __forceinline__ void ring_step(const RingCtx<D> &c, char *ring, int b,
                                          StageRegs<D> &regs, const bf16x8 (&qv)[D / 32],
                                          float scale_log2, int lane, RowState<D> &st) {
  using R = Ring<D>;
  stage_store<D>(ring + ST * R::kStage + c.dst0, lane, regs);
  stage_load<D>(tile_of<D>(c, b + kStages), c.voff, regs);
  __syncthreads();
  if (b == c.prio_end_b) __builtin_amdgcn_s_setprio(0);
  if (c.active) {
    const int t0 = c.sb + b * kBlockKeys;
    const bool full = t0 + kBlockKeys <= min(c.ctx, c.se);
    ring_compute<D, NE>(c.ring, ST * R::kStage, c.rl, c.vb, lane, t0, c.se, c.row_limit, full,
                        qv, scale_log2, st);
  }
}

// Steps S .. kStages-1 of one round of the block loop (one step per ring
// stage, the stage index a compile-time constant); true once the sub-piece's
// last block has been computed.
template <int D, int NE, int S>
struct RingRound {
  static __device__ __forceinline__ bool run(const RingCtx<D> &c, char *ring, int b,
                                             StageRegs<D> (&r)[kStages],
                                             const bf16x8 (&qv)[D / 32], float scale_log2,
                                             int lane, RowState<D> &st) {
    ring_step<D, NE, S>(c, ring, b + S, r[S], qv, scale_log2, lane, st);
    if (b + S + 1 >= c.nblk) return true;
    return RingRound<D, NE, S + 1>::run(c, ring, b, r, qv, scale_log2, lane, st);
  }
};
template <int D, int NE>
struct RingRound<D, NE, kStages> {
  static __device__ __forceinline__ bool run(const RingCtx<D> &, char *, int,
                                             StageRegs<D> (&)[kStages],
                                             const bf16x8 (&)[D / 32], float, int,
                                             RowState<D> &) {
    return false;
  }
};

// All blocks of one sub-piece through the ring.
template <int D, int NE>
__device__ __forceinline__ void ring_run(const RingCtx<D> &c, char *ring,
                                         const bf16x8 (&qv)[D / 32], float scale_log2, int lane,
                                         RowState<D> &st) {
  // issued in block order (the empty asm keeps the compiler from reordering
  // them), so that each step waits only for its own block
  StageRegs<D> r[kStages];
#pragma unroll
  for (int s = 0; s < kStages; ++s) {
    stage_load<D>(tile_of<D>(c, s), c.voff, r[s]);
    asm volatile("" ::: "memory");
  }
  // the loop leaves only when a round reports the last block, so every path
  // back to its head has issued the same loads in the same order and the
  // compiler can wait for exactly the block each step writes
  for (int b = 0;; b += kStages)
    if (RingRound<D, NE, 0>::run(c, ring, b, r, qv, scale_log2, lane, st)) break;
  __syncthreads();  // the ring is free for the next sub-piece
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_streamk_kernel(AttnParams p) {
  using R = Ring<D>;
  __shared__ __attribute__((aligned(1024))) char ring[kStages * R::kStage];
  __shared__ int pg[kSubPages + 8];
  __shared__ int lds_plan[2 * kWaves + 8 + kNumPieceCaps * kWaves];

  const Share sh = plan_share(p, lds_plan);
  if (sh.start >= sh.end) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int kq = lane >> 4, n = lane & 15;
  // keys of the share (virtual) run at raised priority; -1: none
  const bool boost = (int)blockIdx.x >= p.num_cu;
  if (boost) __builtin_amdgcn_s_setprio(1);
  const int boost_keys = boost ? (int)((long long)(sh.end - sh.start) * kBoostPct / 100) : -1;

  // this wave's share of every ring load: page parity pp, K (waves 0-1) or V
  const int pp = wave & 1, kind = wave >> 1;
  RingCtx<D> c;
  c.ring = ring;
  c.pg = pg;
  c.pp = pp;
  c.page_bytes = (size_t)2 * p.hkv * kPage * D * sizeof(uint16_t);
  c.dst0 = kind * R::kKRegion + pp * R::kChunks * 1024;
  c.voff = 16u * (uint32_t)(kind == 0 ? k_unit(lane, pp) : v_unit_inv(lane));
  c.rl = ring_lane<D>(lane);

  int i = sh.i, g = sh.g, off = sh.off, pos = sh.start, piece = 0;
  // metadata of the request last read: the next KV head's segment of the
  // same request (the usual next piece) needs no second read of it
  int i_meta = sh.i;
  ReqMeta meta = sh.first;
  while (pos < sh.end && i < p.num_reqs) {
    if (i != i_meta) {
      meta = load_req(p, i);
      i_meta = i;
    }
    const ReqMeta rq = meta;
    if (rq.seg == 0) {  // sentinel or bad metadata: no keys in the plan
      ++i;
      continue;
    }
    // offsets are virtual: the segment's keys follow its lead-in of
    // sh.lead keys (none in the small-batch plan)
    const int segv = rq.seg + sh.lead;
    const int take = min(segv - off, sh.end - pos);
    const int key_begin = max(off - sh.lead, 0);
    const int key_end = min(rq.len, off + take - sh.lead);
    if (key_end <= key_begin) break;  // the share ends inside the lead-in
    const bool complete = off <= sh.lead && off + take == segv;
    const int slot = piece == 0 ? 0 : 1;
    c.kvw = reinterpret_cast<const char *>(p.kv) +
            (size_t)(kind * p.hkv + g) * kPage * D * sizeof(uint16_t);
    c.ctx = rq.ctx;

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
      c.active = rt < nt;
      const int e_lo = ds * ne;
      c.vb = c.rl.v + 512u * (uint32_t)e_lo;
      const int rr = rt * 16 + n;
      const bool valid_row = c.active && rr < rows;
      const int lg = __builtin_ctz(p.group);
      const int j = rr >> lg, hh = rr & (p.group - 1);
      c.row_limit = valid_row ? rq.ctx + j : -1;
      bf16x8 qv[D / 32];
      {
        const uint16_t *qrow =
            p.q + ((size_t)(rq.q0 + j) * p.hq + (size_t)g * p.group + hh) * D;
#pragma unroll
        for (int cc = 0; cc < D / 32; ++cc) {
          uint4 x = make_uint4(0, 0, 0, 0);
          if (valid_row) x = *reinterpret_cast<const uint4 *>(qrow + 32 * cc + 8 * kq);
          qv[cc] = as_bf16x8(x);
        }

      }
      RowState<D> st;
      st.m = -INFINITY;
      st.l = 0.f;
#pragma unroll
      for (int e = 0; e < D / 16; ++e) st.o[e] = f32x4{0.f, 0.f, 0.f, 0.f};

      for (int sb = key_begin; sb < key_end; sb += kSubPages * kPage) {
        const int se = min(key_end, sb + kSubPages * kPage);
        c.sb = sb;
        c.se = se;
        c.nblk = (se - sb + kBlockKeys - 1) / kBlockKeys;
        c.prio_end_b = -1;
        if (boost_keys >= 0) {
          const int left = boost_keys - ((pos - sh.start) + (sb - key_begin));
          c.prio_end_b = left <= 0 ? 0 : (left + kBlockKeys - 1) / kBlockKeys;
        }
        // stage the sub-piece's page ids; an id outside [0, num_pages) breaks
        // the contract and reads page 0 instead (valid memory, result
        // unspecified), pages past the sub-piece read page 0 and are masked
        {
          const int npg = (se - sb + kPage - 1) / kPage;
          const int *pt = p.page_table + (size_t)i * p.max_pages + sb / kPage;
          for (int t = threadIdx.x; t < 2 * c.nblk; t += kThreads) {
            int id = t < npg ? pt[t] : 0;
            pg[t] = (unsigned)id < (unsigned)p.num_pages ? id : 0;
          }
          __syncthreads();
        }
        if (ne == D / 16)
          ring_run<D, D / 16>(c, ring, qv, p.scale_log2, lane, st);
        else if (ne == D / 32)
          ring_run<D, D / 32>(c, ring, qv, p.scale_log2, lane, st);
        else
          ring_run<D, D / 64>(c, ring, qv, p.scale_log2, lane, st);
      }
      if (c.active) write_tile<D>(p, g, complete, slot, rq, rt, e_lo, ne, lane, st.l, st);
    }

    pos += take;
    off += take;
    ++piece;
    if (off == segv) {
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
// Workgroup (x, g, i) owns kCombThreads/(D/4) live rows of request i and KV head g;
// each thread owns 4 output dims of one row and issues the loads of up to 8
// partials at a time.  Workgroups with z == B zero the tail rows instead.
template <int D>
__global__ __launch_bounds__(kCombThreads) void attn_combine_kernel(AttnParams p) {
  constexpr int kLanesPerRow = D / 4;
  constexpr int kRows = kCombThreads / kLanesPerRow;
  const int g = blockIdx.y, i = blockIdx.z;
  const int G = p.group;
  if (i == p.num_reqs) {
    const int live = min(max(p.cu[p.num_reqs], 0), p.cap);
    const int per_row = G * (D / 8);
    const int total = (p.cap - live) * per_row;
    for (int idx = blockIdx.x * kCombThreads + threadIdx.x; idx < total;
         idx += gridDim.x * kCombThreads) {
      const int r = live + idx / per_row, rem = idx % per_row;
      const int hh = rem / (D / 8), d8 = rem % (D / 8);
      uint16_t *o = p.out + ((size_t)r * p.hq + (size_t)g * G + hh) * D + 8 * d8;
      *reinterpret_cast<uint4 *>(o) = make_uint4(0, 0, 0, 0);
    }
    return;
  }
  // Every plan entry and metadata word this workgroup may need, loaded in
  // one round trip: the empty asm uses them all before the first branch,
  // so the compiler cannot sink the loads that one path needs behind the
  // branches (which made a chain of dependent round trips).
  int prefix = p.plan[i], next = p.plan[i + 1];  // p.plan[B] is the total
  int share = p.plan[p.num_reqs + 1];
  int pc_prefix = p.plan[p.num_reqs + 2 + i];  // read by the small-batch plan only
  int cq0 = p.cu[i], cq1 = p.cu[i + 1], cctx = p.ctx[i];
  asm volatile("" : "+s"(prefix), "+s"(next), "+s"(share), "+s"(pc_prefix), "+s"(cq0),
               "+s"(cq1), "+s"(cctx));
  ReqMeta rq;
  rq.q0 = cq0;
  rq.ctx = cctx;
  rq.k = cq1 - cq0;
  rq.len = cctx + rq.k;
  rq.seg = segment_of(p, cq0, cq1, cctx);
  const int seg = next - prefix;
  if (seg <= 0) return;
  const int start = prefix * p.hkv + g * seg;
  const int skew = share > 0 ? share_skew(share) : 0;
  int b0, b1;
  if (share <= 0) {
    // small-batch plan: the segment's n pieces sit on consecutive workgroups,
    // each the first (and only) piece of its workgroup
    const int n = seg_pieces(seg, -share);
    b0 = pc_prefix * p.hkv + g * n;
    b1 = b0 + n - 1;
  } else {
    // stream-K: seg includes the lead-in, and the first workgroup with any
    // of the segment's keys is the one holding the first key after it
    b0 = share_owner(start + kLeadKeys, share, skew);
    b1 = share_owner(start + seg - 1, share, skew);
  }
  if (b0 == b1) return;  // one workgroup held the whole segment
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
    const int slot = share <= 0 || share_begin(b, share, skew) >= start ? 0 : 1;
    return ((size_t)b * 2 + slot) * (G * kMaxQlen) + rr;
  };

  float mx = -INFINITY;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  if (n_parts <= 8) {
    // the common case: every load in one round trip
    float2 l8[8];
    f32x4 o8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool in = u < n_parts;
      const size_t pr = prow(u);
      l8[u] = in ? p.part_ml[pr] : make_float2(-INFINITY, 0.f);
      o8[u] = in ? *reinterpret_cast<const f32x4 *>(p.part_o + pr * D + 4 * d4)
                 : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) mx = fmaxf(mx, l8[u].x);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float w = exp2f(l8[u].x - mx);
      den += w * l8[u].y;
      acc += w * o8[u];
    }
  } else {
    for (int u0 = 0; u0 < n_parts; u0 += 8) {
      float m8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        m8[u] = u0 + u < n_parts ? p.part_ml[prow(u0 + u)].x : -INFINITY;
#pragma unroll
      for (int u = 0; u < 8; ++u) mx = fmaxf(mx, m8[u]);
    }
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
  }
  const float inv = 1.f / den;
  uint2 w2;
  w2.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  w2.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<uint2 *>(p.out + row * D + 4 * d4) = w2;
}

// Compute units of the current device (cached per device; a host query).
int device_cus() {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev] > 0) return cache[dev];
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  cache[dev] = cus;
  return cus;
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
// workgroups (a 256-CU MI355X holds 512 of this kernel at once, two per CU) and never
// more than the 32-key blocks the largest batch could hold.  The workspace
// is sized for it.
int32_t attn_grid_cap(const dsv_attn_dims &d) {
  constexpr long long kMaxGrid = 1024;
  const long long blocks = (long long)d.num_reqs * d.num_kv_heads *
                           ((d.max_kv_len + kBlockKeys - 1) / kBlockKeys);
  return (int32_t)(blocks < kMaxGrid ? blocks : kMaxGrid);
}

int32_t attn_num_cu() { return device_cus(); }

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
  w.part_ml_off = align_up((size_t)(2 * d.num_reqs + 3) * sizeof(int32_t), 256);
  w.part_o_off = align_up(w.part_ml_off + rows * sizeof(float2), 256);
  w.total = align_up(w.part_o_off + rows * d.head_dim * sizeof(float), 256);
  return w;
}

hipError_t launch_verify_attn(const AttnParams &p, int head_dim, hipStream_t s) {
  // rows of one request and KV head: G * k_i <= G * 16
  const int comb_rows = head_dim == 128 ? kCombThreads / 32 : kCombThreads / 16;
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
    hipLaunchKernelGGL(attn_combine_kernel<128>, grid_comb, dim3(kCombThreads), 0, s, p);
  else
    hipLaunchKernelGGL(attn_combine_kernel<64>, grid_comb, dim3(kCombThreads), 0, s, p);
  timing_mark(kTimeAttnCombine, true, s);
  return hipGetLastError();
}

}  // namespace dsv
