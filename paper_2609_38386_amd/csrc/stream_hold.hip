// dlfp_stream_hold: a one-wave kernel that idles on the device wall clock so
// that launches the host enqueues meanwhile reach the GPU back to back.  A
// completion timer started after it then measures device work only, without
// the host's launch gaps (the per-layer latency of an iteration, Sec. 3).
#include <hip/hip_runtime.h>

#include "dlfp.h"

namespace {

__global__ void stream_hold_kernel(unsigned long long ticks, unsigned int max_polls) {
  const unsigned long long t0 = wall_clock64();
  // Bounded twice: by the clock and by a poll count, so a stalled clock still ends.
  for (unsigned int i = 0; i < max_polls; ++i) {
    if (wall_clock64() - t0 >= ticks) break;
    __builtin_amdgcn_s_sleep(8);
  }
}

}  // namespace

extern "C" int dlfp_stream_hold(int32_t microseconds, hipStream_t stream) {
  if (microseconds < 1 || microseconds > DLFP_MAX_HOLD_US) return DLFP_EINVAL;
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DLFP_EHIP;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      khz <= 0)
    return DLFP_EHIP;
  const unsigned long long ticks = (unsigned long long)khz * (unsigned long long)microseconds / 1000ull;
  // One s_sleep 8 lasts about 512 cycles (~0.2 us), so 100 polls per microsecond
  // covers the wait with a wide margin and still ends within ~20x its length.
  const unsigned int max_polls = 100u * (unsigned int)microseconds;
  hipLaunchKernelGGL(stream_hold_kernel, dim3(1), dim3(64), 0, stream, ticks, max_polls);
  return hipGetLastError() == hipSuccess ? DLFP_OK : DLFP_EHIP;
}
