// accept.hip -- greedy acceptance for gfx950: per-row vocabulary argmax
// followed by the longest-prefix compare against the drafted tokens.
//
// What it computes (Sec. III-D "Prefix verifier" at temperature 0, where the
// target policy is one-hot at its argmax; Sec. I defines the accepted tokens
// as the contiguous candidate prefix, anchor excluded): t_r = argmax of live
// row r (lowest index on ties); a_i = length of the prefix of candidates
// with t_{o+j} == draft[o+j+1]; the successor is t_{o+a_i}.
//
// How: the logits stream is the whole cost (2 bytes per element at bf16),
// so the argmax runs on (vocabulary chunk x row) workgroups, each streaming
// 16 KiB with 16-byte coalesced loads issued back to back, reducing
// (value, index) pairs inside the wave with DPP moves and across the
// four waves in LDS, and writing one pair per (row, chunk).  No atomics: a
// second kernel, one wave per request, reduces the chunk pairs in a fixed
// order and does the prefix compare with a ballot.  The comparison is exact
// (bf16 and fp32 widen exactly to fp32), so the result is bit-exact and
// independent of scheduling.
#include "dsv_internal.h"

#include <math.h>

#include <mutex>

// Scratch of the no-allocation entry point (dsv_accept_noalloc): the chunk
// maxima live here instead of in a caller workspace.  Each GPU the library
// runs on holds its own copy until the process ends.  In host code this name
// is a host-side stand-in, not a device address: host code only ever uses the
// address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[DSV_ACCEPT_NOALLOC_MAX_BYTES];

namespace dsv {
namespace {

constexpr int kThreads = 256;

// (v1, i1) beats (v2, i2): larger value, or equal value and lower index.
// Equal compares +0 and -0 as equal, as the definition requires.
__device__ __forceinline__ bool better(float v1, int i1, float v2, int i2) {
  return v1 > v2 || (v1 == v2 && i1 < i2);
}

__device__ __forceinline__ void take(float &bv, int &bi, float v, int i) {
  if (better(v, i, bv, bi)) {
    bv = v;
    bi = i;
  }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <bool kBf16>
__device__ __forceinline__ float elem(const void *row, int v) {
  if (kBf16) return __uint_as_float((uint32_t)((const uint16_t *)row)[v] << 16);
  return ((const float *)row)[v];
}

// Best (value, index) pair of a wave, in lane 63, with DPP moves instead of
// shuffles (which compile to LDS permutes): exchanges inside quads, then
// the half-row and row mirrors, then the row broadcasts.  A lane whose row
// the broadcast skips keeps its own pair (a no-op take).  `better` is a
// total order, so the pairing does not change the result.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ void dpp_take(float &bv, int &bi) {
  const int ov = __builtin_amdgcn_update_dpp(__float_as_int(bv), __float_as_int(bv), kCtrl,
                                             kRowMask, 0xf, false);
  const int oi = __builtin_amdgcn_update_dpp(bi, bi, kCtrl, kRowMask, 0xf, false);
  take(bv, bi, __int_as_float(ov), oi);
}

__device__ __forceinline__ void wave_best(float &bv, int &bi) {
  dpp_take<0xB1, 0xf>(bv, bi);   // quad_perm [1,0,3,2]
  dpp_take<0x4E, 0xf>(bv, bi);   // quad_perm [2,3,0,1]
  dpp_take<0x141, 0xf>(bv, bi);  // row_half_mirror
  dpp_take<0x140, 0xf>(bv, bi);  // row_mirror
  dpp_take<0x142, 0xa>(bv, bi);  // row_bcast:15 into rows 1 and 3
  dpp_take<0x143, 0xc>(bv, bi);  // row_bcast:31 into rows 2 and 3
}

// One 16-byte vector starting at element `base` (VEC elements).
template <bool kBf16>
__device__ __forceinline__ void take_vec(u32x4 x, int base, float &bv, int &bi) {
  if (kBf16) {
    const uint32_t w[4] = {x[0], x[1], x[2], x[3]};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      take(bv, bi, bf16_lo(w[q]), base + 2 * q);
      take(bv, bi, bf16_hi(w[q]), base + 2 * q + 1);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) take(bv, bi, __uint_as_float(x[q]), base + q);
  }
}

template <bool kBf16>
__global__ __launch_bounds__(kThreads) void argmax_chunk_kernel(
    const void *logits, const int32_t *cu, int32_t num_reqs, int32_t cap,
    int32_t vocab, int32_t num_chunks, float *best_val, int32_t *best_idx) {
  constexpr int kEs = kBf16 ? 2 : 4;         // bytes per element
  constexpr int kVec = 16 / kEs;             // elements per 16-byte load
  constexpr int kUnroll = kAcceptChunk / (kThreads * kVec);
  const int c = blockIdx.x, r = blockIdx.y;
  const int live = min(cu[num_reqs], cap);
  if (r >= live) return;

  const char *row = (const char *)logits + (size_t)r * vocab * kEs;
  const int begin = c * kAcceptChunk;
  const int end = min(vocab, begin + kAcceptChunk);
  float bv = -INFINITY;
  int bi = 0x7FFFFFFF;

  // scalar head up to 16-byte alignment, vector body, scalar tail
  const uintptr_t addr = (uintptr_t)(row + (size_t)begin * kEs);
  const int head = min(end - begin, (int)(((16 - (addr & 15)) & 15) / kEs));
  const int vb = begin + head;
  const int nvec = (end - vb) / kVec;
  const int ve = vb + nvec * kVec;
  const int tid = threadIdx.x;
  if (tid < head) take(bv, bi, elem<kBf16>(row, begin + tid), begin + tid);
  if (tid < end - ve) take(bv, bi, elem<kBf16>(row, ve + tid), ve + tid);
  const u32x4 *vp = (const u32x4 *)(row + (size_t)vb * kEs);
  if (nvec == kThreads * kUnroll) {
    u32x4 x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) x[u] = __builtin_nontemporal_load(vp + u * kThreads + tid);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) take_vec<kBf16>(x[u], vb + (u * kThreads + tid) * kVec, bv, bi);
  } else {
    for (int q = tid; q < nvec; q += kThreads)
      take_vec<kBf16>(__builtin_nontemporal_load(vp + q), vb + q * kVec, bv, bi);
  }

  // wave reduction (the result lands in lane 63), then across the four
  // waves through LDS
  wave_best(bv, bi);
  __shared__ float sv[kThreads / kWave];
  __shared__ int si[kThreads / kWave];
  const int wave = tid / kWave, lane = tid % kWave;
  if (lane == kWave - 1) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    bv = sv[0];
    bi = si[0];
    for (int w = 1; w < kThreads / kWave; ++w) take(bv, bi, sv[w], si[w]);
    best_val[(size_t)r * num_chunks + c] = bv;
    best_idx[(size_t)r * num_chunks + c] = bi;
  }
}

// One wave per request: lane j reduces row o+j over the chunks (in chunk
// order), the ballot of mismatches gives the accepted length.
__global__ __launch_bounds__(kWave) void prefix_kernel(
    const int32_t *cu, const int32_t *draft, int32_t *accept_len,
    int32_t *next_token, int32_t num_reqs, int32_t cap, int32_t num_chunks,
    const float *best_val, const int32_t *best_idx) {
  const int i = blockIdx.x, lane = threadIdx.x;
  const int o = cu[i], k = cu[i + 1] - o;
  if (k == 0) {
    if (lane == 0) {
      accept_len[i] = 0;
      next_token[i] = -1;
    }
    return;
  }
  if (k < 0 || k > kMaxQlen || o < 0 || o + k > cap) return;  // bad metadata
  // the drafted token each row is compared with, loaded with the chunk pairs
  const int want = lane < k - 1 ? draft[o + lane + 1] : -1;
  int t = -1;
  if (lane < k) {
    // the row's chunk pairs in chunk order, loaded kBatch at a time so that
    // the loads of a batch are in flight together (one batch up to 32
    // chunks, a 262,144-token vocabulary)
    constexpr int kBatch = 32;
    const size_t base = (size_t)(o + lane) * num_chunks;
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
    for (int c0 = 0; c0 < num_chunks; c0 += kBatch) {
      float v[kBatch];
      int x[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int c = min(c0 + u, num_chunks - 1);  // clamped: repeats are harmless
        v[u] = best_val[base + c];
        x[u] = best_idx[base + c];
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) take(bv, bi, v[u], x[u]);
    }
    t = bi;
  }
  const bool mismatch = lane < k - 1 && t != want;
  const unsigned long long mask = __ballot(mismatch);
  const int a = mask ? __builtin_ctzll(mask) : k - 1;
  const int succ = __builtin_amdgcn_readlane(t, a);  // a is uniform (from the ballot)
  if (lane == 0) {
    accept_len[i] = a;
    next_token[i] = succ;
  }
}

}  // namespace

// Device address of the no-allocation scratch on the current device,
// resolved once per device with that device current (nullptr on failure).
void *accept_noalloc_scratch() {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    addr[dev] = p;
  }
  return addr[dev];
}

AcceptWorkspace accept_workspace_layout(int32_t cap, int32_t vocab) {
  AcceptWorkspace w;
  w.num_chunks = (vocab + kAcceptChunk - 1) / kAcceptChunk;
  const size_t n = (size_t)cap * w.num_chunks;
  w.val_off = 0;
  w.idx_off = align_up(n * sizeof(float), 256);
  w.total = align_up(w.idx_off + n * sizeof(int32_t), 256);
  return w;
}

hipError_t launch_accept(const void *logits, int dtype, const int32_t *cu,
                         const int32_t *draft, int32_t *accept_len,
                         int32_t *next_token, int32_t num_reqs, int32_t cap,
                         int32_t vocab, float *best_val, int32_t *best_idx,
                         int32_t num_chunks, hipStream_t s) {
  const dim3 grid(num_chunks, cap);
  timing_mark(kTimeArgmax, false, s);
  if (dtype == DSV_BF16)
    hipLaunchKernelGGL(argmax_chunk_kernel<true>, grid, dim3(kThreads), 0, s, logits,
                       cu, num_reqs, cap, vocab, num_chunks, best_val, best_idx);
  else
    hipLaunchKernelGGL(argmax_chunk_kernel<false>, grid, dim3(kThreads), 0, s, logits,
                       cu, num_reqs, cap, vocab, num_chunks, best_val, best_idx);
  timing_mark(kTimeArgmax, true, s);
  timing_mark(kTimePrefix, false, s);
  hipLaunchKernelGGL(prefix_kernel, dim3(num_reqs), dim3(kWave), 0, s, cu, draft,
                     accept_len, next_token, num_reqs, cap, num_chunks, best_val,
                     best_idx);
  timing_mark(kTimePrefix, true, s);
  return hipGetLastError();
}

}  // namespace dsv
