// predictor.hip -- acceptance-predictor forward for gfx950.
//
// What it computes (Sec. III-C, Eqs. (4)-(5)): for every live request of a
// bucket, predLogits = relu(features . W1 + b1) . W2 + b2, a perceptron with
// one ReLU hidden layer of 64 units (the paper's 1735 -> 64 -> 15).  Rows
// past the live count get zeros.
//
// How: the first layer is a small GEMM, [N x in_dim] x [in_dim x 64], split
// over K so that each workgroup reads its slice of W1 once for a tile of up
// to 64 requests: the W1 slice and the feature tile go to LDS, and each
// thread accumulates one hidden unit for 16 requests, reading features as
// LDS broadcasts.  Partial sums go to a workspace in
// slice order; a second kernel, one wave per request, adds them in that
// order with b1, applies the ReLU and evaluates the output layer.  fp32
// throughout and deterministic.
#include "dsv_internal.h"

namespace dsv {
namespace {

constexpr int kH = kPredHidden;  // hidden units (one per lane)
constexpr int kKT = 64;          // features per K slice
constexpr int kRT = 64;          // requests per tile
constexpr int kThreads = 256;
constexpr int kRowsPerThread = kRT / (kThreads / kH);  // 16
constexpr int kLdsStride = kKT + 4;                     // keeps float4 rows aligned

__device__ __forceinline__ int live_count(const int32_t *num_live, int n_bs) {
  const int n = *num_live;
  return n < 0 ? 0 : (n > n_bs ? n_bs : n);
}

__global__ __launch_bounds__(kThreads) void mlp_hidden_partial_kernel(
    const float *features, const int32_t *num_live, const float *w1, float *part,
    int32_t n_bs, int32_t in_dim) {
  __shared__ __align__(16) float sf[kRT][kLdsStride];  // feature tile [request][k]
  __shared__ float sw[kKT][kH];                         // W1 slice [k][hidden unit]
  const int ks = blockIdx.x, r0 = blockIdx.y * kRT, tid = threadIdx.x;
  const int n = live_count(num_live, n_bs);
  if (r0 >= n) return;  // no live row in this tile: its partials are never read
  const int k0 = ks * kKT;
  // W1 slice (rows of 64 contiguous weights) and the feature tile, zero past
  // the last feature and the live rows: every load is issued before the
  // first LDS store (clamped addresses instead of branches)
  constexpr int kPer = kKT * kH / kThreads;  // 16 of each per thread
  float wv[kPer], fv[kPer];
#pragma unroll
  for (int it = 0; it < kPer; ++it) {
    const int idx = tid + it * kThreads;
    const int k = k0 + idx / kH;
    wv[it] = w1[(size_t)(k < in_dim ? k : in_dim - 1) * kH + idx % kH];
    const int row = r0 + idx / kKT, kf = k0 + idx % kKT;
    const bool ok = row < n && kf < in_dim;
    fv[it] = features[ok ? (size_t)row * in_dim + kf : 0];
  }
#pragma unroll
  for (int it = 0; it < kPer; ++it) {
    const int idx = tid + it * kThreads;
    sw[idx / kH][idx % kH] = k0 + idx / kH < in_dim ? wv[it] : 0.f;
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
  const int n = live_count(num_live, n_bs);
  if (i >= n) {
    for (int j = lane; j < out_dim; j += kWave) out[(size_t)i * out_dim + j] = 0.f;
    return;
  }
  // slice partials in slice order, eight loads in flight at a time
  float hsum = 0.f;
  int s = 0;
  for (; s + 8 <= n_slices; s += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = part[((size_t)(s + q) * n_bs + i) * kH + lane];
#pragma unroll
    for (int q = 0; q < 8; ++q) hsum += v[q];
  }
  for (; s < n_slices; ++s) hsum += part[((size_t)s * n_bs + i) * kH + lane];
  hsum += b1[lane];
  sh[lane] = hsum > 0.f ? hsum : 0.f;
  __syncthreads();
  for (int j = lane; j < out_dim; j += kWave) {
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
  const dim3 grid(slices, (n_bs + kRT - 1) / kRT);
  timing_mark(kTimePredictor, false, s);
  hipLaunchKernelGGL(mlp_hidden_partial_kernel, grid, dim3(kThreads), 0, s, features,
                     num_live, w1, part, n_bs, in_dim);
  hipLaunchKernelGGL(mlp_output_kernel, dim3(n_bs), dim3(kWave), 0, s, part, num_live, b1, w2,
                     b2, out, n_bs, slices, out_dim);
  const hipError_t e = hipGetLastError();
  timing_mark(kTimePredictor, true, s);
  return e;
}

}  // namespace dsv
