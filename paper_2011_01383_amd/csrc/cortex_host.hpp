// Host-side helpers shared by the entry points: knobs, co-residency limits and
// the cooperative launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cortex.h"

namespace cortex {

int64_t knob(int32_t which);
void set_last_grid(int which, int32_t grid);

// Ticks of the 100 MHz wall clock (s_memrealtime) for the barrier spin limit.
inline uint64_t barrier_timeout_ticks() {
  int64_t us = knob(CORTEX_KNOB_BARRIER_TIMEOUT_US);
  if (us < 0) us = 0;
  return (uint64_t)us * 100u;
}

// Largest grid of `kernel` (block threads, dynamic LDS) that can be co-resident.
template <typename Kernel>
int max_coresident(Kernel kernel, int threads, size_t dyn_lds) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, dyn_lds) != hipSuccess) return -1;
  return cus * per_cu;
}

inline int num_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

// Cooperative launch of a persistent kernel whose single argument is a struct.
template <typename Kernel, typename Args>
int launch_coop(Kernel kernel, int grid, int threads, size_t dyn_lds, const Args &args, void *stream) {
  void *kargs[] = {(void *)&args};
  hipError_t e = hipLaunchCooperativeKernel((const void *)kernel, dim3(grid), dim3(threads), kargs,
                                            (unsigned int)dyn_lds, (hipStream_t)stream);
  if (e == hipErrorCooperativeLaunchTooLarge) return CORTEX_E_TOO_LARGE;
  return e == hipSuccess ? CORTEX_OK : CORTEX_E_HIP;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace cortex
