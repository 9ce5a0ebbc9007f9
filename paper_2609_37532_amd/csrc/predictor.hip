// predictor.hip -- acceptance-predictor forward for gfx950.
//
// What it computes (Sec. III-C, Eqs. (4)-(5)): for every live request of a
// bucket, predLogits = relu(features . W1 + b1) . W2 + b2, a perceptron with
// one ReLU hidden layer of 64 units (the paper's 1735 -> 64 -> 15).  Rows
// past the live count get zeros.
//
// How: the first layer is a small GEMM, [N x in_dim] x [in_dim x 64], split
// over K so that each workgroup reads its slice of W1 once for a tile of 16,
// 32 or 64 requests (the smallest that holds the bucket, up to 64): the W1
// slice and the feature tile go to LDS, and each thread accumulates one
// hidden unit for a quarter of the tile's requests, reading features as
// LDS broadcasts.  Partial sums go to a workspace in
// slice order; a second kernel, one wave per request, adds them in that
// order with b1, applies the ReLU and evaluates the output layer.  Each
// kernel issues its loads in one round trip, ahead of the live count they
// do not depend on.  fp32 throughout and deterministic.
#include "dsv_internal.h"

namespace dsv {
namespace {

constexpr int kH = kPredHidden;  // hidden units (one per lane)
constexpr int kKT = 64;          // features per K slice
constexpr int kThreads = 256;
constexpr int kRowGroups = kThreads / kH;  // 4: one per wave
constexpr int kLdsStride = kKT + 4;        // keeps float4 rows aligned

// Requests per tile: 16, 32 or 64, the smallest that holds the bucket (up
// to 64), so a small bucket does not multiply zero rows.
int tile_rows(int n_bs) { return n_bs <= 16 ? 16 : (n_bs <= 32 ? 32 : 64); }

__device__ __forceinline__ int live_count(const int32_t *num_live, int n_bs) {
  const int n = *num_live;
  return n < 0 ? 0 : (n > n_bs ? n_bs : n);
}

template <int kRT>
__global__ __launch_bounds__(kThreads) void mlp_hidden_partial_kernel(
    const float *features, const int32_t *num_live, const float *w1, float *part,
    int32_t n_bs, int32_t in_dim) {
  constexpr int kRowsPerThread = kRT / kRowGroups;
  __shared__ __align__(16) float sf[kRT][kLdsStride];  // feature tile [request][k]
  __shared__ float sw[kKT][kH];                         // W1 slice [k][hidden unit]
  const int ks = blockIdx.x, r0 = blockIdx.y * kRT, tid = threadIdx.x;
  if (r0 >= n_bs) return;
  const int k0 = ks * kKT;
  // W1 slice (rows of 64 contiguous weights), the feature tile and the live
  // count, all loaded together: the feature rows are the tile's rows of the
  // bucket (clamped addresses, every one inside [N_bs][in_dim]), and rows
  // past the live count and columns past in_dim are zeroed in LDS
  constexpr int kPerW = kKT * kH / kThreads;   // 16 weights per thread
  constexpr int kPerF = kRT * kKT / kThreads;  // 4, 8 or 16 features per thread
  float wv[kPerW], fv[kPerF];
#pragma unroll
  for (int it = 0; it < kPerW; ++it) {
    const int idx = tid + it * kThreads;
    const int k = k0 + idx / kH;
    wv[it] = w1[(size_t)(k < in_dim ? k : in_dim - 1) * kH + idx % kH];
  }
#pragma unroll
  for (int it = 0; it < kPerF; ++it) {
    const int idx = tid + it * kThreads;
    const int row = r0 + idx / kKT, kf = k0 + idx % kKT;
    fv[it] = features[(size_t)(row < n_bs ? row : n_bs - 1) * in_dim +
                      (kf < in_dim ? kf : in_dim - 1)];
  }
  const int n = live_count(num_live, n_bs);
  if (r0 >= n) return;  // no live row in this tile: its partials are never read
#pragma unroll
  for (int it = 0; it < kPerW; ++it) {
    const int idx = tid + it * kThreads;
    sw[idx / kH][idx % kH] = k0 + idx / kH < in_dim ? wv[it] : 0.f;
  }
#pragma unroll
  for (int it = 0; it < kPerF; ++it) {
    const int idx = tid + it * kThreads;
    const int row = r0 + idx / kKT, kf = k0 + idx % kKT;
    sf[idx / kKT][idx % kKT] = (row < n && kf < in_dim) ? fv[it] : 0.f;
  }
  __syncthreads();
  // thread: hidden unit h for 16 requests; features are LDS broadcasts
  // (every lane of a wave reads the same row)
  const int h = tid % kH, rg = tid / kH;
  float acc[kRowsPerThread];
#pragma unroll
  for (int q = 0; q < kRowsPerThread; ++q) acc[q] = 0.f;
  for (int kk = 0; kk < kKT; kk += 4) {
    const float w0 = sw[kk][h], w1v = sw[kk + 1][h], w2v = sw[kk + 2][h], w3 = sw[kk + 3][h];
#pragma unroll
    for (int q = 0; q < kRowsPerThread; ++q) {
      const float4 fv = *reinterpret_cast<const float4 *>(&sf[rg * kRowsPerThread + q][kk]);
      acc[q] += fv.x * w0 + fv.y * w1v + fv.z * w2v + fv.w * w3;
    }
  }
#pragma unroll
  for (int q = 0; q < kRowsPerThread; ++q) {
    const int row = r0 + rg * kRowsPerThread + q;
    if (row < n) part[((size_t)ks * n_bs + row) * kH + h] = acc[q];
  }
}

__global__ __launch_bounds__(kWave) void mlp_output_kernel(
    const float *part, const int32_t *num_live, const float *b1, const float *w2,
    const float *b2, float *out, int32_t n_bs, int32_t n_slices, int32_t out_dim) {
  __shared__ float sh[kH];
  const int i = blockIdx.x, lane = threadIdx.x;
  // Everything the row needs is loaded before the live count is known (the
  // addresses do not depend on it): the slice partials of hidden unit
  // `lane` (all of them at once up to kSlicesAtOnce slices), b1, and the W2
  // column and b2 of output `lane`.  A row past the live count reads stale
  // partials and discards them.
  constexpr int kSlicesAtOnce = 32;
  const bool all_at_once = n_slices <= kSlicesAtOnce;
  float v[kSlicesAtOnce];
#pragma unroll
  for (int q = 0; q < kSlicesAtOnce; ++q)
    v[q] = all_at_once && q < n_slices ? part[((size_t)q * n_bs + i) * kH + lane] : 0.f;
  const float b1v = b1[lane];
  const int j0 = lane;
  const bool col0 = j0 < out_dim;
  float wc0[kH];
#pragma unroll
  for (int u = 0; u < kH; ++u) wc0[u] = w2[(size_t)u * out_dim + (col0 ? j0 : 0)];
  const float b2v = b2[col0 ? j0 : 0];
  const int n = live_count(num_live, n_bs);
  if (i >= n) {
    for (int j = lane; j < out_dim; j += kWave) out[(size_t)i * out_dim + j] = 0.f;
    return;
  }
  // slice partials added in slice order
  float hsum = 0.f;
  if (all_at_once) {
#pragma unroll
    for (int q = 0; q < kSlicesAtOnce; ++q)
      if (q < n_slices) hsum += v[q];
  } else {
    int s = 0;
    for (; s + 8 <= n_slices; s += 8) {
      float w[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = part[((size_t)(s + q) * n_bs + i) * kH + lane];
#pragma unroll
      for (int q = 0; q < 8; ++q) hsum += w[q];
    }
    for (; s < n_slices; ++s) hsum += part[((size_t)s * n_bs + i) * kH + lane];
  }
  hsum += b1v;
  sh[lane] = hsum > 0.f ? hsum : 0.f;
  __syncthreads();
  if (col0) {
    float o = 0.f;
#pragma unroll
    for (int u = 0; u < kH; ++u) o += sh[u] * wc0[u];
    out[(size_t)i * out_dim + j0] = o + b2v;
  }
  for (int j = lane + kWave; j < out_dim; j += kWave) {
    float wc[kH];
#pragma unroll
    for (int u = 0; u < kH; ++u) wc[u] = w2[(size_t)u * out_dim + j];
    float o = 0.f;
#pragma unroll
    for (int u = 0; u < kH; ++u) o += sh[u] * wc[u];
    out[(size_t)i * out_dim + j] = o + b2[j];
  }
}

}  // namespace

size_t predictor_workspace_bytes(int32_t n_bs, int32_t in_dim) {
  const size_t slices = (size_t)((in_dim + kKT - 1) / kKT);
  return align_up(slices * (size_t)n_bs * kH * sizeof(float), 256);
}

hipError_t launch_predictor(const float *features, const int32_t *num_live, const float *w1,
                            const float *b1, const float *w2, const float *b2, float *out,
                            int32_t n_bs, int32_t in_dim, int32_t out_dim, float *part,
                            hipStream_t s) {
  const int slices = (in_dim + kKT - 1) / kKT;
  const int rt = tile_rows(n_bs);
  const dim3 grid(slices, (n_bs + rt - 1) / rt);
  timing_mark(kTimePredictor, false, s);
  if (rt == 16)
    hipLaunchKernelGGL(mlp_hidden_partial_kernel<16>, grid, dim3(kThreads), 0, s, features,
                       num_live, w1, part, n_bs, in_dim);
  else if (rt == 32)
    hipLaunchKernelGGL(mlp_hidden_partial_kernel<32>, grid, dim3(kThreads), 0, s, features,
                       num_live, w1, part, n_bs, in_dim);
  else
    hipLaunchKernelGGL(mlp_hidden_partial_kernel<64>, grid, dim3(kThreads), 0, s, features,
                       num_live, w1, part, n_bs, in_dim);
  hipLaunchKernelGGL(mlp_output_kernel, dim3(n_bs), dim3(kWave), 0, s, part, num_live, b1, w2,
                     b2, out, n_bs, slices, out_dim);
  const hipError_t e = hipGetLastError();
  timing_mark(kTimePredictor, true, s);
  return e;
}

}  // namespace dsv
