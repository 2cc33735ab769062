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

int num_cus();
int cached_occupancy(const void *kernel, int threads, size_t dyn_lds = 0);

// Largest grid of `kernel` (block threads, no dynamic LDS) that can be co-resident.
template <typename Kernel>
int max_coresident(Kernel kernel, int threads) {
  const int cus = num_cus();
  const int per_cu = cached_occupancy((const void *)kernel, threads, 0);
  if (cus <= 0 || per_cu <= 0) return -1;
  return cus * per_cu;
}

// Launch of a persistent kernel whose single argument is a struct.  A grid of
// at most one workgroup per CU is launched plainly: on a GPU that is not
// shared with other work every workgroup is resident at once, and a barrier
// wait that never completes (a GPU shared with other persistent work) ends at
// its spin limit with CORTEX_ST_BARRIER_TIMEOUT instead of hanging.  Larger
// grids, or CORTEX_KNOB_COOPERATIVE = 1, use the cooperative launch, which
// guarantees co-residency at a higher launch cost.
template <typename Kernel, typename Args>
int launch_persistent(Kernel kernel, int grid, int threads, size_t dyn_lds, const Args &args, void *stream) {
  void *kargs[] = {(void *)&args};
  hipError_t e;
  if (knob(CORTEX_KNOB_COOPERATIVE) == 0 && grid <= num_cus()) {
    e = hipLaunchKernel((const void *)kernel, dim3(grid), dim3(threads), kargs, dyn_lds, (hipStream_t)stream);
  } else {
    e = hipLaunchCooperativeKernel((const void *)kernel, dim3(grid), dim3(threads), kargs,
                                   (unsigned int)dyn_lds, (hipStream_t)stream);
    if (e == hipErrorCooperativeLaunchTooLarge) return CORTEX_E_TOO_LARGE;
  }
  return e == hipSuccess ? CORTEX_OK : CORTEX_E_HIP;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Where a forward launch keeps its workspace header, its tagged staging of h
// and of the second state, and the TreeGRU phase values.
struct FwdRegions {
  void *header;
  void *hs, *cs;
  float *keep;
};

// Internal entry points shared by the C entry points (dry_run: every host
// check, nothing enqueued).
int linearize_impl(const int32_t *d_children, int32_t N, int32_t K, const cortex_lin_t *lin, int32_t *d_status,
                   void *d_ws, size_t ws_bytes, void *stream, bool dry_run);
int tree_infer_impl(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                    const float *d_x_table, int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                    const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status, void *lin_ws,
                    size_t lin_ws_bytes, void *fwd_ws, size_t fwd_ws_bytes, const FwdRegions *fixed, void *stream,
                    bool dry_run);
bool fixed_regions(int32_t cell, int32_t N, int32_t H, void *header, size_t header_cap, void *hs, size_t hs_cap,
                   void *cs, size_t cs_cap, void *keep, size_t keep_cap, FwdRegions &out);
size_t forward_header_bytes();

}  // namespace cortex
