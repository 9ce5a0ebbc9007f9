// timing.hip -- HIP-event kernel timing for measurement harnesses.
#include "dsv_internal.h"

#include <vector>

namespace dsv {
namespace {

struct Timing {
  bool on = false;
  int capacity = 0;        // launch records available
  int used = 0;            // records completed
  int open_kind = -1;      // kind of the launch whose start was recorded
  std::vector<hipEvent_t> start, stop;
  std::vector<int> kind;
};

Timing &timing() {
  static Timing t;
  return t;
}

void release(Timing &t) {
  for (hipEvent_t e : t.start) (void)hipEventDestroy(e);
  for (hipEvent_t e : t.stop) (void)hipEventDestroy(e);
  t.start.clear();
  t.stop.clear();
  t.kind.clear();
  t.capacity = t.used = 0;
  t.open_kind = -1;
  t.on = false;
}

}  // namespace

void timing_mark(int kind, bool end, hipStream_t s) {
  Timing &t = timing();
  if (!t.on) return;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
  if (!end) {
    if (t.used >= t.capacity) return;
    if (hipEventRecord(t.start[t.used], s) == hipSuccess) t.open_kind = kind;
  } else if (t.open_kind == kind) {
    if (hipEventRecord(t.stop[t.used], s) == hipSuccess) {
      t.kind[t.used] = kind;
      ++t.used;
    }
    t.open_kind = -1;
  }
}

}  // namespace dsv

using namespace dsv;

extern "C" {

int dsv_timing_start(int32_t max_launches) {
  if (max_launches < 1 || max_launches > (1 << 20)) return DSV_ERR_DIMS;
  Timing &t = timing();
  release(t);
  t.start.resize(max_launches);
  t.stop.resize(max_launches);
  t.kind.assign(max_launches, -1);
  // Timing-only events: recording them does no system-scope fence, so the
  // interval does not include a writeback and invalidation of the caches
  // (the kernel's own end-of-dispatch release is still inside it).
  constexpr unsigned kFlags = hipEventDisableSystemFence;
  for (int n = 0; n < max_launches; ++n) {
    if (hipEventCreateWithFlags(&t.start[n], kFlags) != hipSuccess ||
        hipEventCreateWithFlags(&t.stop[n], kFlags) != hipSuccess) {
      t.start.resize(n);
      t.stop.resize(n);
      release(t);
      return DSV_ERR_HIP;
    }
  }
  t.capacity = max_launches;
  t.on = true;
  return DSV_OK;
}

int dsv_timing_stop(float *total_ms, int32_t *launches) {
  if (!total_ms || !launches) return DSV_ERR_NULL;
  Timing &t = timing();
  for (int k = 0; k < DSV_TIMING_KINDS; ++k) {
    total_ms[k] = 0.f;
    launches[k] = 0;
  }
  int rc = DSV_OK;
  for (int n = 0; n < t.used; ++n) {
    float ms = 0.f;
    if (hipEventSynchronize(t.stop[n]) != hipSuccess ||
        hipEventElapsedTime(&ms, t.start[n], t.stop[n]) != hipSuccess) {
      rc = DSV_ERR_HIP;
      continue;
    }
    const int k = t.kind[n];
    if (k >= 0 && k < DSV_TIMING_KINDS) {
      total_ms[k] += ms;
      launches[k] += 1;
    }
  }
  release(t);
  return rc;
}

int dsv_timing_stop_each(float *ms, int32_t *kinds, int32_t capacity, int32_t *count) {
  if (!ms || !kinds || !count) return DSV_ERR_NULL;
  if (capacity < 0) return DSV_ERR_DIMS;
  Timing &t = timing();
  int rc = DSV_OK, n_out = 0;
  for (int n = 0; n < t.used && n_out < capacity; ++n) {
    float v = 0.f;
    if (hipEventSynchronize(t.stop[n]) != hipSuccess ||
        hipEventElapsedTime(&v, t.start[n], t.stop[n]) != hipSuccess) {
      rc = DSV_ERR_HIP;
      continue;
    }
    ms[n_out] = v;
    kinds[n_out] = t.kind[n];
    ++n_out;
  }
  *count = n_out;
  release(t);
  return rc;
}

}  // extern "C"
