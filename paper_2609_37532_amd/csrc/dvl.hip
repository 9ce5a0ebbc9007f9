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
// How: one workgroup, one thread per request slot (N_bs <= 1024).  The
// one-at-a-time loop of Eq. (9) is replaced by an equivalent selection.
// Because scores never increase along a block, the loop visits the
// candidate slots in a fixed total order: for growing, by score descending,
// then request ascending, then position ascending; for shrinking, by score
// ascending, then request ascending, then position descending.  Closing a
// gap of g therefore takes exactly the first g candidates of that order, and
// the candidates each request takes form a prefix of its own list.  The
// g-th candidate's score is found with a most-significant-digit-first radix
// select over the binary32 bit patterns (four 8-bit passes, histograms in
// LDS; scores are non-negative so their bit patterns order like the values,
// and the shrink case complements them); requests then take every candidate
// that beats it plus their share of the candidates equal to it, handed out
// in request order by an exclusive scan.  Work is O(W) per thread per pass
// instead of |gap| <= 7N serial argmax steps.  Packing runs one thread per
// packed row, finding its request by binary search over the offsets in LDS,
// so the stores are coalesced.
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

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int t = __shfl_up(v, d, kWave);
    if (lane >= d) v += t;
  }
  return v;
}

// Exclusive prefix sum over the workgroup in thread order; *total receives
// the sum.  Every thread of the block must call it (it synchronises).
__device__ int block_excl_scan(int v, int *s_wave, int *total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int incl = wave_incl_scan(v, lane);
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  int base = 0, sum = 0;
  for (int i = 0; i < nw; ++i) {
    const int t = s_wave[i];
    base += i < wave ? t : 0;
    sum += t;
  }
  __syncthreads();  // s_wave is reused by the next scan
  *total = sum;
  return base + incl - v;
}

__global__ __launch_bounds__(kMaxReqs) void dvl_kernel(DvlArgs a) {
  __shared__ int32_t s_off[kMaxReqs + 1];
  __shared__ uint32_t s_hist[256];
  __shared__ int32_t s_wave[kMaxWaves];
  __shared__ uint32_t s_sel[2];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int w = a.w;
  int n = *a.num_live;
  n = n < 0 ? 0 : (n > a.n_bs ? a.n_bs : n);
  const int m_live = (w / 2) * n;
  const int m_bs = (w / 2) * a.n_bs;
  const bool live = tid < n;

  // ---- prefix scores and initial length (Eqs. (6)-(7))
  float q[kMaxW];
  q[0] = 1.f;
#pragma unroll
  for (int j = 1; j < kMaxW; ++j) q[j] = 0.f;
  int k0 = 0;
  if (live) {
    const float *row = a.pred_logits + (size_t)tid * (w - 1);
#pragma unroll
    for (int j = 1; j < kMaxW; ++j) {
      if (j < w) {
        const float s = score_of(row[j - 1]);
        q[j] = s < q[j - 1] ? s : q[j - 1];  // a NaN score keeps the minimum
      }
    }
    float ell = 0.f;
#pragma unroll
    for (int j = 1; j < kMaxW; ++j)
      if (j < w) ell += q[j];
    const float r = floorf(ell + 0.5f);
    k0 = r < 1.f ? 1 : (r > (float)w ? w : (int)r);
  }
  if (a.scores && tid < a.n_bs) {
    float *dst = a.scores + (size_t)tid * w;
#pragma unroll
    for (int j = 0; j < kMaxW; ++j)
      if (j < w) dst[j] = live ? q[j] : 0.f;
  }

  // ---- budget gap and the equivalent of the one-slot-at-a-time loop (Eq. (9))
  int seed_sum;
  (void)block_excl_scan(k0, s_wave, &seed_sum);
  const int gap = m_live - seed_sum;  // uniform across the workgroup
  int change = 0;
  if (gap != 0) {
    const bool grow = gap > 0;
    uint32_t key[kMaxW];
    uint32_t valid = 0;
#pragma unroll
    for (int j = 0; j < kMaxW; ++j) {
      const uint32_t b = __float_as_uint(q[j]);
      key[j] = grow ? b : ~b;
      const bool cand = grow ? (j >= k0 && j < w) : (j >= 1 && j < k0);
      valid |= (live && cand) ? (1u << j) : 0u;
    }
    uint32_t want = (uint32_t)(grow ? gap : -gap);  // rank of the last slot taken
    uint32_t prefix = 0;
    if (tid == 0) s_sel[0] = s_sel[1] = 0;
#pragma unroll
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int b = tid; b < 256; b += blockDim.x) s_hist[b] = 0;
      __syncthreads();
      const uint32_t hi = shift == 24 ? 0u : (0xFFFFFFFFu << (shift + 8));
#pragma unroll
      for (int j = 0; j < kMaxW; ++j)
        if (((valid >> j) & 1u) && (key[j] & hi) == (prefix & hi))
          atomicAdd(&s_hist[(key[j] >> shift) & 255u], 1u);
      __syncthreads();
      if (tid < kWave) {
        // lane L holds digits 255-4L .. 252-4L (descending key order)
        uint32_t h[4];
        int local = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          h[c] = s_hist[255 - 4 * lane - c];
          local += (int)h[c];
        }
        const int incl = wave_incl_scan(local, lane);
        const uint32_t excl = (uint32_t)(incl - local);
        if (excl < want && want <= (uint32_t)incl) {
          uint32_t cum = excl;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            if (want <= cum + h[c]) {
              s_sel[0] = prefix | ((uint32_t)(255 - 4 * lane - c) << shift);
              s_sel[1] = want - cum;
              break;
            }
            cum += h[c];
          }
        }
      }
      __syncthreads();
      prefix = s_sel[0];
      want = s_sel[1];
    }
    // prefix = the key of the last candidate taken; want = how many of the
    // candidates with exactly that key are taken (in request order)
    int gt = 0, eq = 0;
#pragma unroll
    for (int j = 0; j < kMaxW; ++j) {
      if ((valid >> j) & 1u) {
        gt += key[j] > prefix ? 1 : 0;
        eq += key[j] == prefix ? 1 : 0;
      }
    }
    int eq_total;
    const int eq_before = block_excl_scan(eq, s_wave, &eq_total);
    int take = (int)want - eq_before;
    take = take < 0 ? 0 : (take > eq ? eq : take);
    change = grow ? gt + take : -(gt + take);
  }
  const int k = live ? k0 + change : 0;

  // ---- offsets (Eq. (10)); sentinels end up with k = 0 at offset M_live
  int total;
  const int off = block_excl_scan(k, s_wave, &total);
  if (tid < a.n_bs) {
    a.k_out[tid] = k;
    a.cu[tid] = off;
    s_off[tid] = off;
  }
  if (tid == 0) {
    a.cu[a.n_bs] = total;
    s_off[a.n_bs] = total;
  }
  __syncthreads();

  // ---- packing (Eq. (11)) and tail placeholders
  const int live_rows = total < m_bs ? total : m_bs;
  const int ref0 = a.kv_refs[0];
  for (int s = tid; s < m_bs; s += blockDim.x) {
    int t = 0, p = 0, r = ref0;
    if (s < live_rows) {
      int lo = 0, hi = n - 1;  // largest request with s_off <= s
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= s) lo = mid;
        else hi = mid - 1;
      }
      const size_t src = (size_t)lo * w + (s - s_off[lo]);
      t = a.tokens[src];
      p = a.positions[src];
      r = a.kv_refs[src];
    }
    a.ptok[s] = t;
    a.ppos[s] = p;
    a.pref[s] = r;
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
  const int threads = ((n_bs + kWave - 1) / kWave) * kWave;
  timing_mark(kTimeDvl, false, s);
  hipLaunchKernelGGL(dvl_kernel, dim3(1), dim3(threads), 0, s, a);
  const hipError_t e = hipGetLastError();
  timing_mark(kTimeDvl, true, s);
  return e;
}

}  // namespace dsv
