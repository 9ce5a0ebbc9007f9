// dvl.hip -- DVL budget allocation and flat-buffer packing for gfx950.
//
// What it computes (Sec. III-C, Alg. 1, Eqs. (6)-(11)): prefix scores as the
// running minimum of the predictor's sigmoids with the anchor fixed at one,
// initial lengths from the rounded score sums, the budget adjustment of
// Eq. (9) (grow the best next slot / shrink the worst last slot, one slot at
// a time, lowest request index on ties), prefix-sum offsets, and the packed
// token, position and cache-reference rows with sentinels and tail
// placeholders.  The paper runs the adjustment inside one GPU block; so does
// this kernel.
//
// How: one workgroup of at least N_bs threads (N_bs <= 1024).  The work is
// latency-bound, so it is spread over every thread of the block: the
// (request, draft position) elements are shared evenly for the sigmoids
// (double precision, the costly part) and for the selection below, and one
// thread per request does the running minimum, the seed and its final
// length.  The one-at-a-time loop of Eq. (9) is replaced by an equivalent
// selection.  Because scores never increase along a block, the loop visits
// the candidate slots in a fixed total order: for growing, by score
// descending, then request ascending, then position ascending; for
// shrinking, by score ascending, then request ascending, then position
// descending.  Closing a gap of g therefore takes exactly the first g
// candidates of that order, and the candidates each request takes form a
// prefix of its own list.  The g-th candidate's score is found with a
// most-significant-digit-first radix select over the binary32 bit patterns
// (histograms in LDS; scores are non-negative so their bit patterns order
// like the values, and the shrink case complements them); every candidate
// above it is taken, plus the first of those equal to it in request order,
// counted by an exclusive scan.  Packing runs one thread per packed row,
// reading its request from an owner map in LDS, so the stores are coalesced.
#include "dsv_internal.h"

#include <math.h>

namespace dsv {
namespace {

constexpr int kMaxW = DSV_MAX_QLEN;
constexpr int kMaxReqs = DSV_DVL_MAX_REQS;
constexpr int kMaxWaves = kMaxReqs / kWave;

struct DvlArgs {
  const float *pred_logits;  // [n_bs][w-1]
  const int32_t *num_live;   // device scalar
  const int32_t *tokens, *positions, *kv_refs;  // [n_bs][w]
  int32_t *k_out;    // [n_bs]
  int32_t *cu;       // [n_bs+1]
  int32_t *ptok, *ppos, *pref;  // [m_bs]
  float *scores;     // [n_bs][w] or null
  int32_t n_bs, w;
};

// Score of one predictor logit: the binary32 rounding of the sigmoid
// evaluated in double precision (Eq. (6)).
__device__ __forceinline__ float score_of(float x) {
  const double e = exp(-(double)x);
  return (float)(1.0 / (1.0 + e));
}

// Inclusive prefix sum over the 64 lanes of a wave: Kogge-Stone inside each
// row of 16 lanes with DPP row shifts, then the row totals carried across
// rows with the row-broadcast forms (lane 15 into rows 1 and 3, lane 31 into
// rows 2 and 3).  Lanes without a source keep the `old` operand, 0.
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

// Exclusive prefix sum over the workgroup in thread order; *total receives
// the sum.  Every thread must call it; each call needs its own `s_wave`
// buffer (it is not re-synchronised after reading).  The wave totals are
// read one per lane and scanned with the same DPP sequence.
__device__ __forceinline__ int block_excl_scan(int v, int *s_wave, int *total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int incl = wave_incl_scan(v);
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  const int t = lane < nw ? s_wave[lane] : 0;
  const int tin = wave_incl_scan(t);
  const int base = wave > 0 ? __builtin_amdgcn_readlane(tin, wave - 1) : 0;
  *total = __builtin_amdgcn_readlane(tin, nw - 1);
  return base + incl - v;
}

__global__ __launch_bounds__(kMaxReqs) void dvl_kernel(DvlArgs a) {
  constexpr int kMaxElems = kMaxReqs * (kMaxW - 1);
  __shared__ float s_val[kMaxElems];   // per element: sigmoid, then prefix score
  __shared__ int32_t s_k0[kMaxReqs];   // seeds
  __shared__ int32_t s_chg[kMaxReqs];  // slots each request gains or gives back
  __shared__ int32_t s_off[kMaxReqs + 1];
  __shared__ uint32_t s_hist[4][256];  // one per radix pass
  __shared__ int32_t s_wave[3][kMaxWaves];
  // packed row -> request, written once the scores are dead
  uint16_t *s_owner = reinterpret_cast<uint16_t *>(s_val);
  static_assert(kMaxW / 2 * kMaxReqs * sizeof(uint16_t) <= sizeof(s_val), "owner map");

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int nthr = blockDim.x;
  const int w = a.w;
  const int wm1 = w - 1;
  const int n_el = a.n_bs * wm1;             // (request, position 1..W-1) elements
  const int per = (n_el + nthr - 1) / nthr;  // elements per thread, <= W-1

  // Issue every load that does not depend on the live count together: this
  // thread's logits (elements tid + u * nthr, coalesced), the count and the
  // placeholder reference.
  float x[kMaxW - 1];
#pragma unroll
  for (int u = 0; u < kMaxW - 1; ++u) {
    if (u < per) {
      const int e = tid + u * nthr;
      x[u] = a.pred_logits[e < n_el ? e : n_el - 1];
    }
  }
  int n = *a.num_live;
  const int ref0 = a.kv_refs[0];
  // keep all of them ahead of the first use: the loads may not pass the
  // first statement, the arithmetic may not pass the second
  asm volatile("" ::: "memory");
#pragma unroll
  for (int u = 0; u < kMaxW - 1; ++u)
    if (u < per) asm volatile("" : "+v"(x[u]));
  n = n < 0 ? 0 : (n > a.n_bs ? a.n_bs : n);
  const int m_live = (w / 2) * n;
  const int m_bs = (w / 2) * a.n_bs;
  for (int b = tid; b < 4 * 256; b += nthr) (&s_hist[0][0])[b] = 0;
  for (int b = tid; b < a.n_bs; b += nthr) s_chg[b] = 0;

  // ---- sigmoids (Eq. (6)), spread over the block
#pragma unroll
  for (int u = 0; u < kMaxW - 1; ++u) {
    if (u < per) {
      const int e = tid + u * nthr;
      if (e < n_el) s_val[e] = score_of(x[u]);
    }
  }
  __syncthreads();

  // ---- running minimum and initial length (Eqs. (6)-(7)), one thread per request
  const bool live = tid < n;
  int k0 = 0;
  if (tid < a.n_bs) {
    float *qrow = s_val + tid * wm1;  // q_1 .. q_{W-1}
    float prev = 1.f, ell = 0.f;
#pragma unroll
    for (int j = 1; j < kMaxW; ++j) {
      if (j < w) {
        const float sig = qrow[j - 1];
        prev = sig < prev ? sig : prev;  // a NaN score keeps the minimum
        qrow[j - 1] = prev;
        ell += prev;
      }
    }
    if (live) {
      const float r = floorf(ell + 0.5f);
      k0 = r < 1.f ? 1 : (r > (float)w ? w : (int)r);
    }
    s_k0[tid] = k0;
    if (a.scores) {
      float *dst = a.scores + (size_t)tid * w;
      dst[0] = live ? 1.f : 0.f;
#pragma unroll
      for (int j = 1; j < kMaxW; ++j)
        if (j < w) dst[j] = live ? qrow[j - 1] : 0.f;
    }
  }

  // ---- budget gap and the equivalent of the one-slot-at-a-time loop (Eq. (9))
  int seed_sum;
  (void)block_excl_scan(k0, s_wave[0], &seed_sum);  // also publishes s_val, s_k0
  const int gap = m_live - seed_sum;  // uniform across the workgroup
  if (gap != 0) {
    const bool grow = gap > 0;
    const uint32_t flip = grow ? 0u : 0xFFFFFFFFu;
    // This thread's elements are e0 .. e0+per-1 (contiguous, in request-major
    // order).  Element (i, j) is a growing candidate if j >= k0_i and a
    // shrinking one if j < k0_i; keys are the score bits, complemented when
    // shrinking, so inside one request they are monotone in j and a thread's
    // candidates sharing the bits above a digit sit next to each other.
    const int e0 = tid * per;
    int ei = e0 / wm1, ej = e0 - ei * wm1 + 1;  // request and position of e0
    uint32_t key[kMaxW - 1];
    int req[kMaxW - 1];
    uint32_t valid = 0;
#pragma unroll
    for (int u = 0; u < kMaxW - 1; ++u) {
      if (u < per) {
        const bool in = e0 + u < n_el;
        const int i = in ? ei : 0;
        const int k0i = s_k0[i];
        key[u] = __float_as_uint(s_val[in ? e0 + u : 0]) ^ flip;
        req[u] = i;
        const bool cand = grow ? (ej >= k0i) : (ej < k0i);
        valid |= (in && i < n && cand) ? (1u << u) : 0u;
        const bool wrap = ej == wm1;
        ei += wrap ? 1 : 0;
        ej = wrap ? 1 : ej + 1;
      }
    }
    uint32_t want = (uint32_t)(grow ? gap : -gap);  // rank of the last slot taken
    // Digits from the top: the exponent bits 23..30 first (bit 31 is the
    // same for every key), then mantissa bits 15..22, 7..14 and 0..6.  The
    // bucket of the want-th key is narrowed pass by pass; once every key in
    // it is taken the remaining passes are skipped.
    uint32_t prefix = flip & 0x80000000u;
    int fshift = 31;
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = pass == 3 ? 0 : 23 - 8 * pass;
      const int width = pass == 3 ? 7 : 8;
      const uint32_t hi = 0xFFFFFFFFu << (shift + width);
      const uint32_t dmask = (1u << width) - 1u;
      uint32_t *hist = s_hist[pass];
      // histogram of the next digit among candidates under the prefix; runs
      // of equal digits are added with one atomic
      uint32_t match = 0;
      uint32_t dig[kMaxW - 1];
#pragma unroll
      for (int u = 0; u < kMaxW - 1; ++u) {
        if (u < per) {
          dig[u] = (key[u] >> shift) & dmask;
          match |= (((valid >> u) & 1u) && (key[u] & hi) == (prefix & hi)) ? (1u << u) : 0u;
        }
      }
      int start = 0;
#pragma unroll
      for (int u = 0; u < kMaxW - 1; ++u) {
        if (u < per) {
          const bool m = (match >> u) & 1u;
          const bool opens =
              m && (u == 0 || !((match >> (u - 1)) & 1u) || dig[u - 1] != dig[u]);
          start = opens ? u : start;
          const bool closes = m && (u + 1 == per || !((match >> (u + 1)) & 1u) ||
                                    dig[u + 1 < kMaxW - 1 ? u + 1 : u] != dig[u]);
          if (closes) atomicAdd(&hist[dig[u]], (uint32_t)(u - start + 1));
        }
      }
      __syncthreads();
      // every wave finds the digit holding the want-th largest key (lane L
      // covers digits 255-4L .. 252-4L, in descending order); the next pass
      // uses another histogram, so no second barrier is needed
      uint32_t h[4];
      int local = 0;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        h[c] = hist[255 - 4 * lane - c];
        local += (int)h[c];
      }
      const int incl = wave_incl_scan(local);
      const uint32_t excl = (uint32_t)(incl - local);
      const bool mine = excl < want && want <= (uint32_t)incl;
      uint32_t dsel = 0, wsel = 0, hsel = 0, cum = excl;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (mine && wsel == 0 && want <= cum + h[c]) {
          dsel = (uint32_t)(255 - 4 * lane - c);
          wsel = want - cum;
          hsel = h[c];
        }
        cum += h[c];
      }
      const unsigned long long bal = __ballot(mine);
      const int src = bal ? (int)__builtin_ctzll(bal) : 0;
      prefix |= (uint32_t)__builtin_amdgcn_readlane((int)dsel, src) << shift;
      want = (uint32_t)__builtin_amdgcn_readlane((int)wsel, src);
      fshift = shift;
      if (want == (uint32_t)__builtin_amdgcn_readlane((int)hsel, src)) break;  // uniform
    }
    // The bucket is the keys that agree with prefix from bit fshift up: every
    // key above it is taken, and the first `want` keys inside it in element
    // (request-major) order -- all of them unless the bucket is one value.
    int eq = 0;
#pragma unroll
    for (int u = 0; u < kMaxW - 1; ++u)
      if (u < per && ((valid >> u) & 1u))
        eq += (key[u] >> fshift) == (prefix >> fshift) ? 1 : 0;
    int eq_total;
    int rank = block_excl_scan(eq, s_wave[1], &eq_total);
    // per-request totals of taken elements, one atomic per run of a request
    int run_i = -1, run_n = 0;
#pragma unroll
    for (int u = 0; u < kMaxW - 1; ++u) {
      if (u < per && ((valid >> u) & 1u)) {
        const bool above = (key[u] >> fshift) > (prefix >> fshift);
        const bool inb = (key[u] >> fshift) == (prefix >> fshift);
        const bool taken = above || (inb && (uint32_t)rank < want);
        rank += inb ? 1 : 0;
        if (req[u] != run_i) {
          if (run_n != 0) atomicAdd(&s_chg[run_i], run_n);
          run_i = req[u];
          run_n = 0;
        }
        run_n += taken ? 1 : 0;
      }
    }
    if (run_n != 0) atomicAdd(&s_chg[run_i], run_n);
    __syncthreads();
  }
  const int change = (tid < a.n_bs && gap != 0) ? s_chg[tid] : 0;
  const int k = live ? k0 + (gap > 0 ? change : -change) : 0;

  // ---- offsets (Eq. (10)); sentinels end up with k = 0 at offset M_live
  int total;
  const int off = block_excl_scan(k, s_wave[2], &total);
  if (tid < a.n_bs) {
    a.k_out[tid] = k;
    a.cu[tid] = off;
    s_off[tid] = off;
  }
  if (tid == 0) {
    a.cu[a.n_bs] = total;
    s_off[a.n_bs] = total;
  }
#pragma unroll
  for (int j = 0; j < kMaxW; ++j)
    if (j < k && off + j < m_bs) s_owner[off + j] = (uint16_t)tid;
  __syncthreads();

  // ---- packing (Eq. (11)) and tail placeholders.  Each thread owns rows
  // tid + u * nthr (at most W/2 of them, as the block has at least N_bs
  // threads).  Sources are resolved first, then all loads are issued, then
  // all stores; a placeholder row loads row 0 and discards it.
  const int live_rows = total < m_bs ? total : m_bs;
  int src[kMaxW / 2];
#pragma unroll
  for (int u = 0; u < kMaxW / 2; ++u) {
    const int s = tid + u * nthr;
    if (s < live_rows) {
      const int i = s_owner[s];
      src[u] = i * w + (s - s_off[i]);
    } else {
      src[u] = -1;
    }
  }
  int tv[kMaxW / 2], pv[kMaxW / 2], rv[kMaxW / 2];
#pragma unroll
  for (int u = 0; u < kMaxW / 2; ++u) {
    const int i = src[u] < 0 ? 0 : src[u];
    tv[u] = a.tokens[i];
    pv[u] = a.positions[i];
    rv[u] = a.kv_refs[i];
  }
#pragma unroll
  for (int u = 0; u < kMaxW / 2; ++u) {
    const int s = tid + u * nthr;
    if (s < m_bs) {
      const bool real = src[u] >= 0;
      a.ptok[s] = real ? tv[u] : 0;
      a.ppos[s] = real ? pv[u] : 0;
      a.pref[s] = real ? rv[u] : ref0;
    }
  }
}

}  // namespace

hipError_t launch_dvl(const float *pred_logits, const int32_t *num_live,
                      const int32_t *tokens, const int32_t *positions,
                      const int32_t *kv_refs, int32_t *k_out, int32_t *cu,
                      int32_t *ptok, int32_t *ppos, int32_t *pref, float *scores,
                      int32_t n_bs, int32_t w, hipStream_t s) {
  DvlArgs a{pred_logits, num_live, tokens, positions, kv_refs, k_out, cu,
            ptok, ppos, pref, scores, n_bs, w};
  // one thread per request slot and, up to the workgroup limit, per packed row
  const int m_bs = (w / 2) * n_bs;
  const int want = m_bs > n_bs ? (m_bs < kMaxReqs ? m_bs : kMaxReqs) : n_bs;
  const int threads = ((want + kWave - 1) / kWave) * kWave;
  timing_mark(kTimeDvl, false, s);
  hipLaunchKernelGGL(dvl_kernel, dim3(1), dim3(threads), 0, s, a);
  const hipError_t e = hipGetLastError();
  timing_mark(kTimeDvl, true, s);
  return e;
}

}  // namespace dsv
