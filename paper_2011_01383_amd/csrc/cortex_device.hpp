// Device-side building blocks shared by the linearizer and the forward kernels:
// the status word, a device-wide barrier for persistent cooperative launches,
// and the fp32 MFMA tile step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cortex.h"

namespace cortex {

// ---------------------------------------------------------------------------
// Workspace header of a persistent launch.
//   line 0, word 0    the barrier generation (written by workgroup 0 only)
//   line 0, word 16   the staging epoch: the tag of the last forward launch on
//                     this workspace that ended normally (see launch tags below)
//   arrive[kMaxGrid]  one arrival word per workgroup (written by its owner only)
//   slot[2][kMaxGrid] per-workgroup values a kernel exchanges between barriers,
//                     double-buffered by round parity (x2 for two values)
//   entered[kMaxGrid] the tag each workgroup of the current forward launch read
// Nothing here needs resetting between launches: barrier epochs are derived
// from the generation, which only grows, so old arrival words never match a
// future epoch.  After a launch that ends with a non-zero status the caller
// must zero the workspace again (the abort can leave arrival words ahead, and
// the staging epoch is not advanced).
// ---------------------------------------------------------------------------
constexpr int kMaxGrid = 4096;
constexpr int kEpochWord = 16;
constexpr size_t kSyncBytes = 128 + sizeof(unsigned int) * (size_t)kMaxGrid * (1 + 4 + 1);

struct SyncWords {
  unsigned int *base;
  __device__ unsigned int *gen() const { return base; }
  __device__ unsigned int *epoch() const { return base + kEpochWord; }
  __device__ unsigned int *arrive(int b) const { return base + 32 + b; }
  // value v (0 or 1) of round parity p for workgroup b
  __device__ unsigned int *slot(int v, int p, int b) const {
    return base + 32 + kMaxGrid + ((v * 2 + p) * kMaxGrid) + b;
  }
  __device__ unsigned int *entered(int b) const { return base + 32 + 5 * kMaxGrid + b; }
};

__device__ __forceinline__ int load_status(const int32_t *status) {
  return __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void raise_status(int32_t *status, int code) {
  // first error wins; later ones are dropped
  int expected = 0;
  __hip_atomic_compare_exchange_strong(status, &expected, code, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned int ld_agent(const unsigned int *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(unsigned int *p, unsigned int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Device-coherent view of a float array written by other workgroups of the
// same launch.  Loads and stores carry the device scope bit (sc1): a store is
// written through to the device coherence point, a load is served from it,
// and neither is satisfied by a CU's L1 or an XCD's L2 copy.  Out-of-range
// offsets read zero and drop stores (buffer bounds check).  Offsets are bytes.
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
constexpr int kScopeDevice = 16;            // buffer cache-policy bit sc1
constexpr int kRawBufferWord3 = 0x00020000;  // 32-bit data format, raw access

struct DevBuf {
  __amdgpu_buffer_rsrc_t r;
  __device__ DevBuf(const float *p, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc((void *)p, (short)0, (int)bytes, kRawBufferWord3)) {}
  __device__ __forceinline__ float4 load4(uint32_t off) const {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kScopeDevice));
  }
  __device__ __forceinline__ u32x4 load4u(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kScopeDevice);
  }
  __device__ __forceinline__ float load1(uint32_t off) const {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kScopeDevice));
  }
  __device__ __forceinline__ void store4(uint32_t off, float4 v) const {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, kScopeDevice);
  }
  __device__ __forceinline__ void store1(uint32_t off, float v) const {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), r, off, 0, kScopeDevice);
  }
};

// Bit casts through a value parameter: clang's __builtin_bit_cast applied
// directly to an ext-vector element (v.z) reads element 0 instead.
__device__ __forceinline__ float as_float(unsigned int u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ unsigned int as_uint(float f) { return __builtin_bit_cast(unsigned int, f); }

// Byte offset beyond every buffer this library builds (sizes are < 2^31):
// a load there returns zeros without touching memory.  Loads whose source is
// absent use it instead of a branch, so they are always issued and their
// results never have to be merged (which would force an early wait).
constexpr uint32_t kNoSource = 0x80000000u;

// ---------------------------------------------------------------------------
// Per-datum ordering between workgroups of one launch (no barrier).  Every
// state element is also staged as an 8-byte (value bits, tag) pair written
// with one device-scope 64-bit store, so a reader sees either an old pair or
// the new one, never half of each.  A launch uses a tag no earlier launch on
// the same workspace used, so a pair carrying the launch's tag is a value
// written by this launch and the staging never needs resetting.  Offsets are
// in bytes; kNoSource reads zeros (tag 0, which no launch uses).
// ---------------------------------------------------------------------------
struct TagBuf {
  __amdgpu_buffer_rsrc_t r;
  __device__ TagBuf(const void *p, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc((void *)p, (short)0, (int)bytes, kRawBufferWord3)) {}
  __device__ __forceinline__ u32x4 load2_at(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kScopeDevice);
  }
  __device__ __forceinline__ u32x2 load1_at(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kScopeDevice);
  }
  // element e
  __device__ __forceinline__ void store1(uint32_t e, float v, uint32_t tag) const {
    u32x2 w;
    w.x = as_uint(v);
    w.y = tag;
    __builtin_amdgcn_raw_buffer_store_b64(w, r, e * 8u, 0, kScopeDevice);
  }
};

// ---------------------------------------------------------------------------
// Launch tags.  A pair in the staging is this launch's value only if no
// earlier launch on the same workspace wrote that tag, so tags come from the
// workspace itself, not from the host: every workgroup reads the staging
// epoch E at entry and uses tag = E + 1 (all workgroups read the same E:
// nothing changes it during the launch), and records that tag in its entered
// word.  At its normal exit workgroup 0 waits until every workgroup of the
// launch has entered, then stores E + 1 as the new epoch, which the next
// launch on the stream reads.  Launches enqueued by different copies of the
// library, or by different processes, on one workspace therefore never reuse
// a tag, as long as they are ordered (the ABI already forbids overlapping
// calls on one workspace).  A zeroed workspace has E = 0 and holds tag 0
// only, which no launch uses; a workspace whose epoch reached 0xFFFFFFFF has
// no tag left and reports CORTEX_ST_EPOCH_WRAP (zero it to continue).  A
// launch that ends with an error does not advance the epoch; the ABI asks for
// the workspace to be zeroed then.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t launch_tag(const unsigned int *sync) {
  return ld_agent(SyncWords{(unsigned int *)sync}.epoch()) + 1u;
}

// After the entry loads: false (and CORTEX_ST_EPOCH_WRAP) when the epoch has
// no tag left; otherwise thread 0 records the workgroup's tag.
__device__ __forceinline__ bool mark_entered(unsigned int *sync, uint32_t tag, int32_t *status) {
  if (tag == 0u) {
    if (threadIdx.x == 0) raise_status(status, CORTEX_ST_EPOCH_WRAP);
    return false;
  }
  if (threadIdx.x == 0) st_agent(SyncWords{sync}.entered(blockIdx.x), tag);
  return true;
}

// At the normal end of a launch that retires its tag, reached by every
// thread of every workgroup: workgroup 0 waits (bounded) for every
// workgroup's entered word, then publishes the tag as the epoch.  Nothing is
// published after an error anywhere in the launch.
__device__ __forceinline__ void retire_tag(unsigned int *sync, uint32_t tag, int32_t *status, uint64_t timeout_ticks) {
  if (blockIdx.x != 0) return;
  const SyncWords sw{sync};
  int ok = 1;
  for (int b = (int)threadIdx.x; b < (int)gridDim.x && ok; b += (int)blockDim.x) {
    const uint64_t t0 = wall_clock64();
    while (ld_agent(sw.entered(b)) != tag) {
      if (load_status(status) != 0) { ok = 0; break; }
      if (wall_clock64() - t0 > timeout_ticks) {
        raise_status(status, CORTEX_ST_BARRIER_TIMEOUT);
        ok = 0;
        break;
      }
    }
  }
  ok = __syncthreads_and(ok);
  if (ok && threadIdx.x == 0 && load_status(status) == 0) st_agent(sw.epoch(), tag);
}

// Read-only input rows (embedding tables, DAG inputs) through the ordinary
// cache hierarchy; out-of-range offsets read zeros.  Offsets are bytes.
struct InBuf {
  __amdgpu_buffer_rsrc_t r;
  __device__ InBuf(const void *p, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc((void *)p, (short)0, (int)bytes, kRawBufferWord3)) {}
  __device__ __forceinline__ u32x4 load4(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  }
  __device__ __forceinline__ unsigned int load1(uint32_t off) const {
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
  }
};

// Makes the compiler complete the load that produced v here (an empty asm
// that reads v).  The memory counter on gfx950 counts stores as well as
// loads, so a wait for a load issued before some stores also waits for those
// stores once they are outstanding; settling a prefetched operand before a
// step's stores keeps its first use from waiting on them.
__device__ __forceinline__ void settle(const u32x4 &v) { asm volatile("" ::"v"(v)); }

__device__ __forceinline__ float4 as_float4(u32x4 v) {
  return make_float4(as_float(v.x), as_float(v.y), as_float(v.z), as_float(v.w));
}

// Wait until every global store this wave issued has completed.  A plain
// __syncthreads() does not do this on gfx950, and the agent-scope release
// below is issued by one wave only.
constexpr int kWaitVmcntZero = 0x0F70;       // s_waitcnt vmcnt(0), other counters not waited on
__device__ __forceinline__ void wave_stores_complete() { __builtin_amdgcn_s_waitcnt(kWaitVmcntZero); }

// ---------------------------------------------------------------------------
// Device-wide barrier for a persistent launch (all workgroups co-resident).
//
// One barrier per level is what the dependence structure needs: no node of a
// level is a child of another node of the same level, so the dependence is
// carried by the level loop only (Appendix A.4).
//
// Lock-free flag barrier: every wave drains its stores, one lane per
// workgroup releases at agent scope (L2 write-back), reads the generation g
// and writes g+1 to its own arrival word.  Workgroup 0 polls all arrival
// words in parallel (one lane per workgroup), then publishes generation g+1;
// the others poll the generation and acquire (L2 invalidate).  No atomic
// read-modify-write is involved, so the cost does not grow with the number
// of workgroups the way a shared arrival counter does (device-scope atomics
// on one address serialise).
//
// kFenced = false is for kernels whose cross-workgroup data all moves through
// DevBuf (device-scope stores and loads): a completed device-scope store is
// already visible at the coherence point, so release reduces to the store
// wait and no L2 write-back or invalidate is needed.
//
// Every wait is bounded by a wall-clock limit; a wait that passes it raises
// CORTEX_ST_BARRIER_TIMEOUT.  A waiter that sees any non-zero status gives up.
// Returns false when the kernel must stop.  With one workgroup it reduces to
// __syncthreads.
// ---------------------------------------------------------------------------
template <bool kFenced = true>
__device__ __forceinline__ bool grid_sync(const SyncWords &sw, int32_t *status, uint64_t timeout_ticks) {
  if (gridDim.x == 1) {
    __syncthreads();
    return load_status(status) == 0;
  }
  __shared__ unsigned int s_gen;
  __shared__ int s_ok;
  wave_stores_complete();
  __syncthreads();
  if (threadIdx.x == 0) {
    if (kFenced) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const unsigned int g = ld_agent(sw.gen());
    s_gen = g;
    s_ok = 1;
    if (blockIdx.x != 0) st_agent(sw.arrive(blockIdx.x), g + 1u);
  }
  __syncthreads();
  const unsigned int g = s_gen;
  if (blockIdx.x == 0) {
    int fail = 0;
    for (int b = 1 + (int)threadIdx.x; b < (int)gridDim.x && !fail; b += (int)blockDim.x) {
      const uint64_t t0 = wall_clock64();
      while (ld_agent(sw.arrive(b)) != g + 1u) {
        if (load_status(status) != 0) { fail = 1; break; }
        if (wall_clock64() - t0 > timeout_ticks) {
          raise_status(status, CORTEX_ST_BARRIER_TIMEOUT);
          fail = 1;
          break;
        }
      }
    }
    if (fail) s_ok = 0;
    __syncthreads();
    if (threadIdx.x == 0) {
      if (kFenced) __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "agent");
      if (s_ok && load_status(status) == 0) {
        st_agent(sw.gen(), g + 1u);
      } else {
        s_ok = 0;
        st_agent(sw.gen(), g + 2u);        // release the waiters; they will see the status
      }
    }
  } else if (threadIdx.x == 0) {
    const uint64_t t0 = wall_clock64();
    int ok = 1;
    while (ld_agent(sw.gen()) == g) {
      if (load_status(status) != 0) { ok = 0; break; }
      if (wall_clock64() - t0 > timeout_ticks) {
        raise_status(status, CORTEX_ST_BARRIER_TIMEOUT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (kFenced) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    if (ok && load_status(status) != 0) ok = 0;
    s_ok = ok;
  }
  __syncthreads();
  return s_ok != 0;
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

// Four output tiles sharing one A fragment: the same four k steps as
// mfma_k16 for each tile, issued step-major so that consecutive MFMAs write
// different accumulators (no back-to-back dependence); every accumulator
// still adds its products in the order mfma_k16 adds them.
template <int NT>
__device__ __forceinline__ void mfma_k16_xn(float4 a4, const float4 (&b4)[NT], floatx4 (&c)[NT]) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) c[nt] = mfma16x16x4(a4.x, b4[nt].x, c[nt]);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) c[nt] = mfma16x16x4(a4.y, b4[nt].y, c[nt]);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) c[nt] = mfma16x16x4(a4.z, b4[nt].z, c[nt]);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) c[nt] = mfma16x16x4(a4.w, b4[nt].w, c[nt]);
}

// Step s (0..3) of mfma_k16_xn alone, so other instructions can be placed
// between the steps; steps 0..3 in order add exactly what mfma_k16_xn adds.
template <int NT>
__device__ __forceinline__ void mfma_kstep_xn(int s, float4 a4, const float4 (&b4)[NT], floatx4 (&c)[NT]) {
  const float a = s == 0 ? a4.x : s == 1 ? a4.y : s == 2 ? a4.z : a4.w;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float b = s == 0 ? b4[nt].x : s == 1 ? b4[nt].y : s == 2 ? b4[nt].z : b4[nt].w;
    c[nt] = mfma16x16x4(a, b, c[nt]);
  }
}

// ---------------------------------------------------------------------------
// Gate nonlinearities from their definitions, on the hardware base-2
// exponential and reciprocal (v_exp_f32, v_rcp_f32, about 1 ulp each):
//   sigmoid(z) = 1 / (1 + e^-z),   tanh(z) = 1 - 2 / (1 + e^2z).
// Overflow of the exponential gives the right limits (1/inf = 0).  The
// absolute error is a few 1e-7 over the whole range; tanh near 0 loses
// relative, not absolute, accuracy to the cancellation.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float exp_fast(float z) { return __builtin_amdgcn_exp2f(z * 1.4426950408889634f); }
__device__ __forceinline__ float sigmoidf(float z) { return __builtin_amdgcn_rcpf(1.0f + exp_fast(-z)); }
__device__ __forceinline__ float tanh_f(float z) {
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + exp_fast(2.0f * z));
}

template <typename T>
__device__ __forceinline__ T ld_nt(const T *p) { return __builtin_nontemporal_load(p); }

}  // namespace cortex
