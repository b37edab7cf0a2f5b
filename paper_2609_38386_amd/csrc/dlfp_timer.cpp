// Completion timer of libdlfp: a pair of HIP events around an iteration's
// device work, read after the work has completed (the latency Eq. 2 is fed,
// Sec. 3.1; completion rather than scheduler-call cadence, Sec. 6.4).
#include <hip/hip_runtime.h>

#include <new>

#include "dlfp.h"

extern "C" {

struct dlfp_timer_s {
  hipEvent_t start, stop;
};

int dlfp_timer_create(dlfp_timer* timer) {
  if (!timer) return DLFP_EINVAL;
  dlfp_timer t = new (std::nothrow) dlfp_timer_s;
  if (!t) return DLFP_EINVAL;
  if (hipEventCreate(&t->start) != hipSuccess) {
    delete t;
    return DLFP_EHIP;
  }
  if (hipEventCreate(&t->stop) != hipSuccess) {
    (void)hipEventDestroy(t->start);
    delete t;
    return DLFP_EHIP;
  }
  *timer = t;
  return DLFP_OK;
}

int dlfp_timer_destroy(dlfp_timer timer) {
  if (!timer) return DLFP_EINVAL;
  const bool ok = hipEventDestroy(timer->start) == hipSuccess &&
                  hipEventDestroy(timer->stop) == hipSuccess;
  delete timer;
  return ok ? DLFP_OK : DLFP_EHIP;
}

int dlfp_timer_start(dlfp_timer timer, hipStream_t stream) {
  if (!timer) return DLFP_EINVAL;
  return hipEventRecord(timer->start, stream) == hipSuccess ? DLFP_OK : DLFP_EHIP;
}

int dlfp_timer_stop(dlfp_timer timer, hipStream_t stream) {
  if (!timer) return DLFP_EINVAL;
  return hipEventRecord(timer->stop, stream) == hipSuccess ? DLFP_OK : DLFP_EHIP;
}

int dlfp_timer_elapsed_ms(dlfp_timer timer, double* ms) {
  if (!timer || !ms) return DLFP_EINVAL;
  if (hipEventSynchronize(timer->stop) != hipSuccess) return DLFP_EHIP;
  float f = 0.f;
  if (hipEventElapsedTime(&f, timer->start, timer->stop) != hipSuccess) return DLFP_EHIP;
  *ms = f;
  return DLFP_OK;
}

}  // extern "C"
