// sample.hip -- stochastic prefix verifier (temperature T > 0) for gfx950.
//
// What it computes (Sec. III-D "Prefix verifier"): the target policy at a
// packed row is P = softmax(logits / T).  Request i's candidates are tested
// in order; candidate x_j = draft[o+j+1] is accepted with probability
// P_{o+j}(x_j), decided by the caller's uniform (accepted iff
// u[o+j][0] < P(x)).  At the first rejection (row o+a) the successor is drawn
// from P_{o+a} with x_a removed and the rest renormalised; if every
// candidate passes, from P_{o+k-1} unchanged.  The draw inverts the
// cumulative distribution in vocabulary order at u[o+a][1].
//
// How: the logits stream is the cost, as for the greedy verifier.  A first
// kernel runs on (vocabulary chunk x live row) workgroups and writes, per
// chunk, the maximum of the scaled logits and the sum of exp2 of their
// differences to it (base-2 exponent with log2(e)/T folded into one
// multiplier).  A second kernel, one workgroup per request, merges those
// pairs into each row's normaliser in chunk order, makes the accept
// decisions from single logit loads, then finds the successor: the chunk
// holding the target mass from the chunk totals, and the token inside it
// with one pass over that chunk and a block scan.  Everything is fp32 and
// deterministic; the decisions agree with exact arithmetic except when a
// uniform lies within rounding of its threshold.
#include "dsv_internal.h"

#include <math.h>

namespace dsv {
namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = kAcceptChunk / kThreads;  // successor-chunk elements per thread

template <bool kBf16>
__device__ __forceinline__ float elem(const void *row, int v) {
  if (kBf16) return __uint_as_float((uint32_t)((const uint16_t *)row)[v] << 16);
  return ((const float *)row)[v];
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// A logit times log2(e)/T, rounded on its own: never fused into a following
// subtraction (a fused multiply-add would skip the product's rounding), so
// every kernel -- and the row maximum -- sees the same value.
__device__ __forceinline__ float scaled(float x, float c) {
#pragma clang fp contract(off)
  return x * c;
}

// Inclusive prefix sum of floats over the 64 lanes of a wave (DPP row shifts,
// then row broadcasts; lanes without a source add 0).  Adding non-negative
// values keeps the prefix non-decreasing, lane by lane.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_add(float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, kRowMask, 0xf, false));
}
__device__ __forceinline__ float wave_incl_scan_f(float v) {
  v += dpp_add<0x111, 0xf>(v);  // row_shr:1
  v += dpp_add<0x112, 0xf>(v);  // row_shr:2
  v += dpp_add<0x114, 0xf>(v);  // row_shr:4
  v += dpp_add<0x118, 0xf>(v);  // row_shr:8
  v += dpp_add<0x142, 0xa>(v);  // row_bcast:15
  v += dpp_add<0x143, 0xc>(v);  // row_bcast:31
  return v;
}

// 2^x with the hardware instruction alone, without the library's denormal
// range handling (a term below 2^-126 of the row maximum contributes
// nothing); every kernel here uses it, so they agree on each term.
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Online (max, sum of exp2(y - max)) accumulation of one scaled value.
__device__ __forceinline__ void acc(float &m, float &s, float y) {
  if (y > m) {
    s = s * fexp2(m - y) + 1.f;
    m = y;
  } else if (y > -INFINITY) {  // a -inf logit adds nothing
    s += fexp2(y - m);
  }
}

__device__ __forceinline__ void merge(float &m, float &s, float om, float os) {
  if (om > m) {
    s = s * fexp2(m - om) + os;
    m = om;
  } else if (om != -INFINITY) {
    s += os * fexp2(om - m);
  }
}

// (max, sum) merge with a DPP-moved partner instead of a shuffle (which
// compiles to an LDS permute).  Lanes that the move skips (row broadcasts
// into masked rows) see the identity (-inf, 0) and stay unchanged.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ void dpp_merge(float &m, float &s) {
  const float om = __int_as_float(__builtin_amdgcn_update_dpp(
      __float_as_int(-INFINITY), __float_as_int(m), kCtrl, kRowMask, 0xf, false));
  const float os = __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(s), kCtrl, kRowMask, 0xf, false));
  merge(m, s, om, os);
}

// Merge over each row of 16 lanes (every lane of the row ends with it):
// exchanges inside quads, then the half-row and row mirrors.
__device__ __forceinline__ void row16_merge(float &m, float &s) {
  dpp_merge<0xB1, 0xf>(m, s);   // quad_perm [1,0,3,2]
  dpp_merge<0x4E, 0xf>(m, s);   // quad_perm [2,3,0,1]
  dpp_merge<0x141, 0xf>(m, s);  // row_half_mirror
  dpp_merge<0x140, 0xf>(m, s);  // row_mirror
}

// Merge over the wave, complete in lane 63: the row merges, then the row
// broadcasts of lane 15 into rows 1 and 3 and of lane 31 into rows 2 and 3.
__device__ __forceinline__ void wave_merge(float &m, float &s) {
  row16_merge(m, s);
  dpp_merge<0x142, 0xa>(m, s);
  dpp_merge<0x143, 0xc>(m, s);
}

template <bool kBf16>
__device__ __forceinline__ void acc_vec(u32x4 x, float c, float &m, float &s) {
  if (kBf16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc(m, s, scaled(bf16_lo(x[q]), c));
      acc(m, s, scaled(bf16_hi(x[q]), c));
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) acc(m, s, scaled(__uint_as_float(x[q]), c));
  }
}

// Per (chunk, live row): max of logits * c and sum of exp2(logits * c - max).
template <bool kBf16>
__global__ __launch_bounds__(kThreads) void softmax_stats_kernel(
    const void *logits, const int32_t *cu, int32_t num_reqs, int32_t cap, int32_t vocab,
    int32_t num_chunks, float c, float *stat_m, float *stat_s) {
  constexpr int kEs = kBf16 ? 2 : 4;
  constexpr int kVec = 16 / kEs;
  constexpr int kUnroll = kAcceptChunk / (kThreads * kVec);
  const int ch = blockIdx.x, r = blockIdx.y;
  const int live = min(cu[num_reqs], cap);
  if (r >= live) return;
  const char *row = (const char *)logits + (size_t)r * vocab * kEs;
  const int begin = ch * kAcceptChunk;
  const int end = min(vocab, begin + kAcceptChunk);
  float m = -INFINITY, s = 0.f;
  const uintptr_t addr = (uintptr_t)(row + (size_t)begin * kEs);
  const int head = min(end - begin, (int)(((16 - (addr & 15)) & 15) / kEs));
  const int vb = begin + head;
  const int nvec = (end - vb) / kVec;
  const int ve = vb + nvec * kVec;
  const int tid = threadIdx.x;
  if (tid < head) acc(m, s, scaled(elem<kBf16>(row, begin + tid), c));
  if (tid < end - ve) acc(m, s, scaled(elem<kBf16>(row, ve + tid), c));
  const u32x4 *vp = (const u32x4 *)(row + (size_t)vb * kEs);
  if (nvec == kThreads * kUnroll) {
    // full chunk: the values sit in registers, so take their maximum first
    // and then one exponential each
    u32x4 x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) x[u] = __builtin_nontemporal_load(vp + u * kThreads + tid);
    constexpr int kN = kUnroll * kVec;
    float y[kN];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (kBf16) {
          y[u * kVec + 2 * q] = scaled(bf16_lo(x[u][q]), c);
          y[u * kVec + 2 * q + 1] = scaled(bf16_hi(x[u][q]), c);
        } else {
          y[u * kVec + q] = scaled(__uint_as_float(x[u][q]), c);
        }
      }
    }
    float lm = y[0];
#pragma unroll
    for (int q = 1; q < kN; ++q) lm = fmaxf(lm, y[q]);
    float ls = 0.f;
    if (lm > -INFINITY) {
#pragma unroll
      for (int q = 0; q < kN; ++q) ls += fexp2(y[q] - lm);
    }
    merge(m, s, lm, ls);
  } else {
    for (int q = tid; q < nvec; q += kThreads)
      acc_vec<kBf16>(__builtin_nontemporal_load(vp + q), c, m, s);
  }
  wave_merge(m, s);  // complete in lane 63
  __shared__ float sm[kThreads / kWave], ss[kThreads / kWave];
  const int wave = tid / kWave, lane = tid % kWave;
  if (lane == kWave - 1) {
    sm[wave] = m;
    ss[wave] = s;
  }
  __syncthreads();
  if (tid == 0) {
    m = sm[0];
    s = ss[0];
    for (int w = 1; w < kThreads / kWave; ++w) merge(m, s, sm[w], ss[w]);
    stat_m[(size_t)r * num_chunks + ch] = m;
    stat_s[(size_t)r * num_chunks + ch] = s;
  }
}

// Chunk statistics kept in LDS for the chunk scan of the drawn row (up to
// this many chunks per row, a 524,288-token vocabulary; beyond it they are
// read again from global memory).
constexpr int kStashChunks = 64;

// One workgroup per request: accept decisions, then the successor draw.
// Everything that does not depend on another load is issued first: the
// chunk statistics of the k rows, the drafted ids with both uniforms of
// each row, and then the logit at each drafted id.
template <bool kBf16>
__global__ __launch_bounds__(kThreads) void stochastic_prefix_kernel(
    const void *logits, const int32_t *cu, const int32_t *draft, const float *uniforms,
    int32_t *accept_len, int32_t *next_token, int32_t num_reqs, int32_t cap, int32_t vocab,
    int32_t num_chunks, float c, const float *stat_m, const float *stat_s) {
  constexpr int kEs = kBf16 ? 2 : 4;
  __shared__ float s_rm[kMaxQlen], s_rz[kMaxQlen];
  __shared__ float s_sm[kMaxQlen][kStashChunks], s_ss[kMaxQlen][kStashChunks];
  __shared__ int s_a, s_removed;
  __shared__ float s_ex, s_u1;
  __shared__ int s_chunk;
  __shared__ float s_target;  // mass still to cover inside the chosen chunk
  __shared__ float s_part[kThreads];  // inclusive token-order sums per thread
  const int i = blockIdx.x, tid = threadIdx.x;
  const int o = cu[i], k = cu[i + 1] - o;
  if (k == 0) {
    if (tid == 0) {
      accept_len[i] = 0;
      next_token[i] = -1;
    }
    return;
  }
  if (k < 0 || k > kMaxQlen || o < 0 || o + k > cap) return;  // bad metadata
  const bool stash = num_chunks <= kStashChunks;

  // wave 0, lane j < k: the drafted id tested at row o+j, both uniforms of
  // the row, and the logit at that id
  int x = -1;
  float u0 = 0.f, u1 = 0.f, lx = 0.f;
  if (tid < k) {
    u0 = uniforms[2 * (size_t)(o + tid)];
    u1 = uniforms[2 * (size_t)(o + tid) + 1];
    if (tid < k - 1) {
      const int d = draft[o + tid + 1];
      x = (d >= 0 && d < vocab) ? d : -1;
    }
  }
  if (x >= 0) lx = elem<kBf16>((const char *)logits + (size_t)(o + tid) * vocab * kEs, x);

  // row normalisers: 16 lanes per row merge that row's chunk pairs in order
  {
    const int j = tid / 16, l = tid % 16;
    float m = -INFINITY, s = 0.f;
    if (j < k) {
      const size_t base = (size_t)(o + j) * num_chunks;
      for (int ch = l; ch < num_chunks; ch += 16) {
        const float cm = stat_m[base + ch], cs = stat_s[base + ch];
        if (stash) {
          s_sm[j][ch] = cm;
          s_ss[j][ch] = cs;
        }
        merge(m, s, cm, cs);
      }
    }
    row16_merge(m, s);
    if (j < k && l == 0) {
      s_rm[j] = m;
      s_rz[j] = s;
    }
  }
  __syncthreads();

  // accept decisions: wave 0, lane j tests candidate j (accepted iff its
  // uniform lies below P(x)); lane a also holds the drawn row's removed
  // token, its unnormalised mass and the draw uniform
  if (tid < kWave) {
    bool reject = false;
    float num = 0.f;
    if (tid < k - 1) {
      if (x >= 0) num = fexp2(scaled(lx, c) - s_rm[tid]);
      reject = !(u0 < num / s_rz[tid]);
    }
    const unsigned long long mask = __ballot(reject);
    const int a = mask ? __builtin_ctzll(mask) : k - 1;
    if (tid == a) {
      s_a = a;
      s_removed = a < k - 1 ? x : -1;
      s_ex = a < k - 1 ? num : 0.f;
      s_u1 = u1;
    }
  }
  __syncthreads();
  const int a = s_a;
  const int r = o + a;
  const char *row = (const char *)logits + (size_t)r * vocab * kEs;
  const float M = s_rm[a];
  const int removed = s_removed;
  const float ex = s_ex;

  // The chunk holding the target mass: wave 0 takes 64 chunks at a time,
  // scans their masses in chunk order and picks the first chunk whose
  // inclusive sum exceeds the target.
  __shared__ int s_alt;  // last chunk with mass other than the removed token's
  if (tid < kWave) {
    const size_t base = (size_t)r * num_chunks;
    const int rc = removed >= 0 ? removed / kAcceptChunk : -1;
    const float t = s_u1 * (s_rz[a] - ex);
    float carry = 0.f;
    int pick = -1, last = -1, alt = -1;
    float pick_rest = 0.f, last_w = 0.f;
    for (int c0 = 0; c0 < num_chunks; c0 += kWave) {
      const int ch = c0 + tid;
      float w = 0.f;
      if (ch < num_chunks) {
        const float sm = stash ? s_sm[a][ch] : stat_m[base + ch];
        const float ss = stash ? s_ss[a][ch] : stat_s[base + ch];
        w = sm == -INFINITY ? 0.f : ss * fexp2(sm - M);
        if (ch == rc) w = fmaxf(w - ex, 0.f);
      }
      const float incl = carry + wave_incl_scan_f(w);
      const unsigned long long pos = __ballot(w > 0.f);
      const unsigned long long other = __ballot(w > 0.f && ch != rc);
      if (pos) {
        last = c0 + 63 - __builtin_clzll(pos);
        last_w = __int_as_float(
            __builtin_amdgcn_readlane(__float_as_int(w), 63 - __builtin_clzll(pos)));
      }
      if (other) alt = c0 + 63 - __builtin_clzll(other);
      const unsigned long long hit = __ballot(w > 0.f && incl > t);
      if (pick < 0 && hit) {
        const int l = __builtin_ctzll(hit);
        const float before =
            l > 0 ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(incl), l - 1)) : carry;
        pick = c0 + l;
        pick_rest = t - before;
      }
      carry = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(incl), kWave - 1));
      if (pick >= 0) break;  // uniform: every lane saw the same ballot
    }
    if (pick < 0) {  // the uniform at or past the rounded total
      pick = last >= 0 ? last : 0;
      pick_rest = last_w;
    }
    if (tid == 0) {
      s_chunk = pick;
      s_target = pick_rest;
      s_alt = alt;
    }
  }
  __syncthreads();

  // Inside the chunk: per-thread masses of 32 consecutive tokens, a block
  // scan in token order, the first thread whose inclusive sum exceeds the
  // target, then the token inside that thread's range.  If rounding left
  // the chosen chunk without mass (only possible for the chunk that held
  // the removed candidate), the last other chunk with mass is used instead,
  // at its end.
  __shared__ float s_wtot[kThreads / kWave];
  __shared__ int s_whit[kThreads / kWave], s_wlast[kThreads / kWave];
  const int wave = tid / kWave, lane = tid % kWave;
  for (int attempt = 0; attempt < 2; ++attempt) {
    const int ch = s_chunk;
    const float t = s_target;
    const int v0 = ch * kAcceptChunk + tid * kPerThread;
    // this thread's run of logits: 16-byte vector loads when the run is
    // whole and aligned (rows of a vocabulary that is a multiple of 8), else
    // element by element
    float x[kPerThread];
    const char *run = row + (size_t)v0 * kEs;
    if (v0 + kPerThread <= vocab && ((uintptr_t)run & 15) == 0) {
      constexpr int kVecs = kPerThread * kEs / 16;
      u32x4 w[kVecs];
#pragma unroll
      for (int u = 0; u < kVecs; ++u) w[u] = reinterpret_cast<const u32x4 *>(run)[u];
#pragma unroll
      for (int u = 0; u < kVecs; ++u)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (kBf16) {
            x[8 * u + 2 * q] = bf16_lo(w[u][q]);
            x[8 * u + 2 * q + 1] = bf16_hi(w[u][q]);
          } else {
            x[4 * u + q] = __uint_as_float(w[u][q]);
          }
        }
    } else {
#pragma unroll
      for (int q = 0; q < kPerThread; ++q)
        x[q] = v0 + q < vocab ? elem<kBf16>(row, v0 + q) : 0.f;
    }
    float e[kPerThread];
    float mine = 0.f;
#pragma unroll
    for (int q = 0; q < kPerThread; ++q) {
      const int v = v0 + q;
      float ev = 0.f;
      if (v < vocab && v != removed) ev = fexp2(scaled(x[q], c) - M);
      e[q] = ev;
      mine += ev;
    }
    float incl = wave_incl_scan_f(mine);
    if (lane == kWave - 1) s_wtot[wave] = incl;
    __syncthreads();
    for (int w = 0; w < wave; ++w) incl += s_wtot[w];
    s_part[tid] = incl;
    const unsigned long long hit = __ballot(mine > 0.f && incl > t);
    const unsigned long long pos = __ballot(mine > 0.f);
    if (lane == 0) {
      s_whit[wave] = hit ? wave * kWave + __builtin_ctzll(hit) : -1;
      s_wlast[wave] = pos ? wave * kWave + 63 - __builtin_clzll(pos) : -1;
    }
    __syncthreads();
    int who = -1, last = -1;
    for (int w = 0; w < kThreads / kWave; ++w) {
      if (who < 0) who = s_whit[w];
      if (s_wlast[w] >= 0) last = s_wlast[w];
    }
    if (who >= 0 || last >= 0) {
      const bool fallback = who < 0;
      if (fallback) who = last;
      if (tid == who) {
        // mass before this thread's range, then the token
        const float before = who > 0 ? s_part[who - 1] : 0.f;
        const float rest = fallback ? mine : t - before;
        float cum = 0.f;
        int pick = -1, lastv = -1;
#pragma unroll
        for (int q = 0; q < kPerThread; ++q) {
          if (e[q] > 0.f) {
            lastv = v0 + q;
            if (pick < 0 && cum + e[q] > rest) pick = v0 + q;
          }
          cum += e[q];
        }
        accept_len[i] = a;
        next_token[i] = pick >= 0 ? pick : lastv;
      }
      return;
    }
    // no mass here: retry at the end of another chunk
    const int alt = s_alt;
    if (attempt == 1 || alt < 0) break;
    __syncthreads();  // every thread has read s_chunk / s_target / s_part
    if (tid == 0) {
      s_chunk = alt;
      s_target = INFINITY;
    }
    __syncthreads();
  }
  // every token but the rejected one has zero probability in fp32: emit the
  // rejected candidate (its renormalised distribution is undefined)
  if (tid == 0) {
    accept_len[i] = a;
    next_token[i] = removed >= 0 ? removed : 0;
  }
}

}  // namespace

SampleWorkspace sample_workspace_layout(int32_t cap, int32_t vocab) {
  SampleWorkspace w;
  w.num_chunks = (vocab + kAcceptChunk - 1) / kAcceptChunk;
  const size_t n = (size_t)cap * w.num_chunks;
  w.m_off = 0;
  w.s_off = align_up(n * sizeof(float), 256);
  w.total = align_up(w.s_off + n * sizeof(float), 256);
  return w;
}

hipError_t launch_accept_stochastic(const void *logits, int dtype, const int32_t *cu,
                                    const int32_t *draft, const float *uniforms,
                                    float scale_log2, int32_t *accept_len,
                                    int32_t *next_token, int32_t num_reqs, int32_t cap,
                                    int32_t vocab, float *stat_m, float *stat_s,
                                    int32_t num_chunks, hipStream_t s) {
  const dim3 grid(num_chunks, cap);
  timing_mark(kTimeSampleStats, false, s);
  if (dtype == DSV_BF16)
    hipLaunchKernelGGL(softmax_stats_kernel<true>, grid, dim3(kThreads), 0, s, logits, cu,
                       num_reqs, cap, vocab, num_chunks, scale_log2, stat_m, stat_s);
  else
    hipLaunchKernelGGL(softmax_stats_kernel<false>, grid, dim3(kThreads), 0, s, logits, cu,
                       num_reqs, cap, vocab, num_chunks, scale_log2, stat_m, stat_s);
  timing_mark(kTimeSampleStats, true, s);
  timing_mark(kTimeSampleDraw, false, s);
  if (dtype == DSV_BF16)
    hipLaunchKernelGGL(stochastic_prefix_kernel<true>, dim3(num_reqs), dim3(kThreads), 0, s,
                       logits, cu, draft, uniforms, accept_len, next_token, num_reqs, cap,
                       vocab, num_chunks, scale_log2, stat_m, stat_s);
  else
    hipLaunchKernelGGL(stochastic_prefix_kernel<false>, dim3(num_reqs), dim3(kThreads), 0, s,
                       logits, cu, draft, uniforms, accept_len, next_token, num_reqs, cap,
                       vocab, num_chunks, scale_log2, stat_m, stat_s);
  timing_mark(kTimeSampleDraw, true, s);
  return hipGetLastError();
}

}  // namespace dsv
