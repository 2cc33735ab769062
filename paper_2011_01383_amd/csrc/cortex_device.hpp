// Device-side building blocks shared by the linearizer and the forward kernels:
// the status word, a device-wide barrier for persistent cooperative launches,
// and the fp32 MFMA tile step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cortex.h"

namespace cortex {

// ---------------------------------------------------------------------------
// Workspace header.  Every persistent launch keeps its synchronisation words at
// the start of the caller's workspace, each in its own 128-byte line.
// ---------------------------------------------------------------------------
struct SyncWords {
  static constexpr int kLine = 32;                 // ints per 128-byte line
  unsigned int *base;
  __device__ unsigned int *count() const { return base; }              // barrier arrivals
  __device__ unsigned int *gen() const { return base + kLine; }        // barrier generation
  __device__ unsigned int *exits() const { return base + 2 * kLine; }  // workgroups finished
  __device__ unsigned int *word(int i) const { return base + (3 + i) * kLine; }  // kernel-specific
};
constexpr size_t kSyncBytes = 16 * 128;            // 16 lines: 3 barrier + 13 kernel words

__device__ __forceinline__ int load_status(const int32_t *status) {
  return __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void raise_status(int32_t *status, int code) {
  // first error wins; later ones are dropped
  int expected = 0;
  __hip_atomic_compare_exchange_strong(status, &expected, code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Device-wide barrier for a cooperative (co-resident) launch.
//
// One barrier per level is what the dependence structure needs: no node of a
// level is a child of another node of the same level, so the dependence is
// carried by the level loop only (Appendix A.4).
//
// Protocol (generation counter): every wave publishes its stores with an
// agent-scope release fence (L2 write-back on gfx950), the workgroup meets at
// s_barrier, then one lane reads the generation, adds itself to the arrival
// count and either (last arriver) resets the count and bumps the generation,
// or spins on the generation with a wall-clock limit.  Every wave then
// acquires at agent scope (L2 invalidate) so the next level reads fresh rows.
//
// A wait that passes its limit raises CORTEX_ST_BARRIER_TIMEOUT; a waiter that
// sees any non-zero status gives up too.  The function returns false when the
// kernel must stop (status set), true otherwise.  With a single workgroup it
// reduces to __syncthreads.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool grid_sync(const SyncWords &sw, int32_t *status, uint64_t timeout_ticks) {
  if (gridDim.x == 1) {
    __syncthreads();
    return load_status(status) == 0;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  __shared__ int s_ok;
  if (threadIdx.x == 0) {
    int ok = 1;
    unsigned int g = __hip_atomic_load(sw.gen(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned int arrived = __hip_atomic_fetch_add(sw.count(), 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (arrived == gridDim.x - 1) {
      __hip_atomic_store(sw.count(), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(sw.gen(), g + 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      const uint64_t t0 = wall_clock64();
      while (__hip_atomic_load(sw.gen(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == g) {
        if (load_status(status) != 0) { ok = 0; break; }
        if (wall_clock64() - t0 > timeout_ticks) {
          raise_status(status, CORTEX_ST_BARRIER_TIMEOUT);
          ok = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (ok && load_status(status) != 0) ok = 0;
    s_ok = ok;
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  return s_ok != 0;
}

// Called by every workgroup as its last action.  The last one to finish
// returns the barrier and the kernel-specific words to zero, so the workspace
// is ready for the next launch even after a timeout.
__device__ __forceinline__ void grid_exit(const SyncWords &sw, int n_words) {
  if (gridDim.x == 1) {
    __syncthreads();
    if (threadIdx.x < (unsigned)n_words) *sw.word(threadIdx.x) = 0u;
    return;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned int done = __hip_atomic_fetch_add(sw.exits(), 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (done == gridDim.x - 1) {
      __hip_atomic_store(sw.count(), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      for (int i = 0; i < n_words; ++i)
        __hip_atomic_store(sw.word(i), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(sw.exits(), 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 MFMA: D(16x16) += A(16x4) * B(4x16), v_mfma_f32_16x16x4_f32.
// Lane l supplies A[l%16][l/16] and B[l/16][l%16]; it receives
// D[4*(l/16) + v][l%16] for v = 0..3.
// ---------------------------------------------------------------------------
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 mfma16x16x4(float a, float b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Accumulate a 16x16 tile over 16 consecutive k: lane (i = l%16, g = l/16)
// holds a4 = A[i][k0+4g .. k0+4g+3] and b4 = B^T[j=i][k0+4g .. +3].  The four
// MFMA steps use k = k0+4g+s for lane group g at step s, a permutation of the
// 16 k values that A and B share, so the sum is unchanged.
__device__ __forceinline__ floatx4 mfma_k16(float4 a4, float4 b4, floatx4 c) {
  c = mfma16x16x4(a4.x, b4.x, c);
  c = mfma16x16x4(a4.y, b4.y, c);
  c = mfma16x16x4(a4.z, b4.z, c);
  c = mfma16x16x4(a4.w, b4.w, c);
  return c;
}

// ---------------------------------------------------------------------------
// Scalar math.  tanhf/expf are the ROCm device-library functions (accurate to
// a few ulp); sigmoid is written from its definition 1/(1+exp(-z)).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float sigmoidf(float z) { return 1.0f / (1.0f + expf(-z)); }
__device__ __forceinline__ float tanh_f(float z) { return tanhf(z); }

template <typename T>
__device__ __forceinline__ T ld_nt(const T *p) { return __builtin_nontemporal_load(p); }

}  // namespace cortex
