// probe.hip -- measurement probe: the HBM read rate of 4 KiB tiles visited
// in a caller-given order.  Not part of the verify path.
//
// A 4 KiB tile is the unit the verify attention reads: one page's keys (or
// values) of one KV head at 16 tokens per page and D = 128 in bf16.  With a
// random visiting order over a pool much larger than the 256 MB Infinity
// Cache, the probe measures the read rate that scattered page tiles can
// reach on the device, the ceiling the attention kernel's streaming phase is
// compared with.  Each workgroup stages its visit ids in LDS, then keeps
// twelve tiles (three 16 KiB blocks) in flight per round, as the attention
// kernel does; the grid size is the caller's, so launch shapes can be swept.
//
// The XOR of every word a workgroup reads goes to sink[workgroup]: the loads
// cannot be dropped, and a test can check the probe read exactly the tiles
// it was given.
#include "dsv_internal.h"

namespace dsv {
namespace {

constexpr int kThreads = 256;
constexpr int kTileBytes = 4096;
constexpr int kTileVecs = kTileBytes / 16;  // one 16-byte vector per thread
constexpr int kInFlight = 12;
static_assert(kTileVecs == kThreads, "one vector per thread per tile");

__global__ __launch_bounds__(kThreads) void read_probe_kernel(
    const u32x4 *buf, int32_t buf_tiles, const int32_t *order, int32_t visits,
    uint32_t *sink) {
  const int per = (int)(((long long)visits + gridDim.x - 1) / gridDim.x);
  const int v0 = (int)min((long long)visits, (long long)blockIdx.x * per);
  const int v1 = min(visits, v0 + per);
  const int tid = threadIdx.x;
  constexpr int kStage = 1024;  // visit ids staged in LDS at a time
  __shared__ int s_id[kStage];
  uint32_t x = 0;
  for (int c0 = v0; c0 < v1; c0 += kStage) {
    const int nc = min(kStage, v1 - c0);
    __syncthreads();  // the previous chunk's ids are no longer read
    for (int t = tid; t < nc; t += kThreads) {
      const int id = order[c0 + t];
      s_id[t] = (unsigned)id < (unsigned)buf_tiles ? id : -1;
    }
    __syncthreads();
    for (int v = 0; v < nc; v += kInFlight) {
      int id[kInFlight];
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) id[u] = v + u < nc ? s_id[v + u] : -1;
      u32x4 d[kInFlight];
#pragma unroll
      for (int u = 0; u < kInFlight; ++u)
        d[u] = id[u] >= 0 ? __builtin_nontemporal_load(buf + (size_t)id[u] * kTileVecs + tid)
                          : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) x ^= d[u][0] ^ d[u][1] ^ d[u][2] ^ d[u][3];
    }
  }
  // XOR across the workgroup: the wave by shuffles, then the four waves
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) x ^= (uint32_t)__shfl_xor((int)x, m, kWave);
  __shared__ uint32_t s[kThreads / kWave];
  if (tid % kWave == 0) s[tid / kWave] = x;
  __syncthreads();
  if (tid == 0) {
    uint32_t t = 0;
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) t ^= s[w];
    sink[blockIdx.x] = t;
  }
}

}  // namespace
}  // namespace dsv

using namespace dsv;

extern "C" int dsv_read_probe(const void *buf, int32_t buf_tiles, const int32_t *order,
                              int32_t visits, uint32_t *sink, int32_t grid,
                              void *hip_stream) {
  if (!buf || !order || !sink) return DSV_ERR_NULL;
  if (buf_tiles < 1 || visits < 1 || grid < 1 || grid > 65535) return DSV_ERR_DIMS;
  if ((uintptr_t)buf & 15u) return DSV_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(read_probe_kernel, dim3(grid), dim3(kThreads), 0,
                     (hipStream_t)hip_stream, (const u32x4 *)buf, buf_tiles, order, visits,
                     sink);
  return hipGetLastError() == hipSuccess ? DSV_OK : DSV_ERR_HIP;
}
