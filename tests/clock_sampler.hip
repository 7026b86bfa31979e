// Test-only measurement library (not part of libtfm): one wave that reads the shader
// clock while other kernels run.  s_memtime counts shader-clock cycles and
// s_memrealtime counts at the fixed wall-clock rate (hipDeviceAttributeWallClockRate),
// so their two differences over a window give the clock the chip ran at.  The wave
// sleeps between reads and stops after a wall-clock window or an iteration cap,
// whichever comes first, so it always exits and takes no issue slots worth noting.
#include <hip/hip_runtime.h>

namespace {

__global__ __launch_bounds__(64) void sample_clock(unsigned long long* out, unsigned long long window_ticks,
                                                   int max_iters) {
  const unsigned long long t0m = __builtin_amdgcn_s_memtime(), t0r = __builtin_amdgcn_s_memrealtime();
  unsigned long long t1m = t0m, t1r = t0r;
  for (int i = 0; i < max_iters; ++i) {
    __builtin_amdgcn_s_sleep(127);
    t1m = __builtin_amdgcn_s_memtime();
    t1r = __builtin_amdgcn_s_memrealtime();
    if (t1r - t0r >= window_ticks) break;
  }
  if (threadIdx.x == 0) {
    out[0] = t1m - t0m;   // shader cycles
    out[1] = t1r - t0r;   // wall-clock ticks
  }
}

}  // namespace

// Enqueue the sampler on `stream` (one wave).  out: 2 device uint64 (cycles, ticks).
// window_ticks: wall-clock ticks to sample for; max_iters: hard cap on the sleep loop
// (each iteration sleeps about 8000 cycles).  Returns 0, or 1 on a launch error.
extern "C" int clock_sampler_launch(unsigned long long* out, unsigned long long window_ticks, int max_iters,
                                    void* stream) {
  hipLaunchKernelGGL(sample_clock, dim3(1), dim3(64), 0, (hipStream_t)stream, out, window_ticks, max_iters);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

// Wall-clock counter rate of the current device in kHz (0 on error).
extern "C" int clock_sampler_wall_khz() {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
  return khz;
}
