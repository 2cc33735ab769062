// Diagnostics: a throughput probe of the fp32 matrix cores, so that achieved
// rates can be set against what the chip sustains, beside its nominal peak;
// and a probe of the fixed cost of ordering one level after another in a
// persistent launch (a device-wide barrier, or the per-datum tagged exchange
// the forward kernels use), which bounds a level loop from below.
#include <atomic>

#include "cortex_device.hpp"
#include "cortex_host.hpp"

namespace cortex {

constexpr int kProbeWaves = 8;          // per workgroup: two per SIMD
constexpr int kProbeChains = 4;         // independent accumulators per wave
constexpr int kProbeSteps = 4;          // dependent MFMAs per chain per iteration

// Every wave runs iters x kProbeChains x kProbeSteps chained 16x16x4 fp32
// MFMAs on register operands; one value per lane is kept so the work stays.
__global__ void __launch_bounds__(64 * kProbeWaves) probe_mfma_kernel(float *sink, int32_t iters, float seed) {
  floatx4 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) acc[c] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float x = seed + (float)threadIdx.x * 1e-7f, y = seed * 0.5f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) {
      acc[c] = mfma16x16x4(x, y, acc[c]);
      acc[c] = mfma16x16x4(y, x, acc[c]);
      acc[c] = mfma16x16x4(x, x, acc[c]);
      acc[c] = mfma16x16x4(y, y, acc[c]);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// ---------------------------------------------------------------------------
// Level-ordering probe: a persistent grid that runs `levels` empty levels.
// Mode 0 ends every level with the device-wide barrier (grid_sync, no cache
// maintenance: the variant kernels use when their data moves through
// device-scope accesses).  Mode 1 orders the levels as the forward kernels
// do, per datum: at each level every workgroup publishes one (value, tag)
// pair with a device-scope store and waits until the pair of every workgroup
// carries that level's tag or a later one, one lane polling per workgroup.
// Each workgroup's pair has a 128-byte line of its own: with 16 workgroups'
// pairs packed into a line, an empty level costs about 50% more (2.6 against
// 1.7 us at 256 workgroups), the stores and polls of a line queuing behind
// each other.
// A workgroup can only run one level ahead of the slowest, so a later tag
// also proves the level was published.  Every wait ends at the spin limit or
// on a non-zero status.  levels = 0 leaves the launch cost alone.
// ---------------------------------------------------------------------------
constexpr int kProbeThreads = 512;       // the forward kernels' workgroup size
constexpr uint32_t kProbeLine = 128;     // bytes per workgroup pair

struct LevelProbeArgs {
  unsigned int *sync;
  void *pairs;
  int32_t *status;
  int32_t levels, mode;
  uint32_t tag0;
  uint64_t timeout;
};

__global__ void __launch_bounds__(kProbeThreads) probe_levels_kernel(LevelProbeArgs a) {
  if (load_status(a.status) != 0) return;
  const TagBuf tb(a.pairs, (uint32_t)gridDim.x * kProbeLine);
  for (int l = 0; l < a.levels; ++l) {
    if (a.mode == 0) {
      if (!grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout)) return;
      continue;
    }
    const uint32_t want = a.tag0 + (uint32_t)l;
    if (threadIdx.x == 0) tb.store1(blockIdx.x * (kProbeLine / 8u), (float)l, want);
    int fail = 0;
    if ((int)threadIdx.x < (int)gridDim.x) {
      const uint32_t off = threadIdx.x * kProbeLine;
      const uint64_t t0 = wall_clock64();
      while ((int)(tb.load1_at(off).y - want) < 0) {
        if (load_status(a.status) != 0) { fail = 1; break; }
        if (wall_clock64() - t0 > a.timeout) {
          raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
          fail = 1;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (__syncthreads_or(fail)) return;
  }
}

constexpr size_t kProbePairsOffset = 256 * ((kSyncBytes + 255) / 256);

}  // namespace cortex

using namespace cortex;

static std::atomic<uint32_t> g_probe_tag{0};

extern "C" size_t cortex_probe_levels_workspace_bytes(void) {
  return kProbePairsOffset + (size_t)kMaxGrid * kProbeLine;
}

extern "C" int cortex_probe_levels(int32_t mode, int32_t grid, int32_t levels, int32_t *d_status, void *d_ws,
                                   size_t ws_bytes, void *stream) {
  const int cus = num_cus();
  if (!d_status || !d_ws || (mode != 0 && mode != 1) || levels < 0 || grid < 1) return CORTEX_E_INVAL;
  if (cus <= 0) return CORTEX_E_HIP;
  if (grid > cus || grid > kMaxGrid) return CORTEX_E_TOO_LARGE;
  if (ws_bytes < cortex_probe_levels_workspace_bytes()) return CORTEX_E_WORKSPACE;
  LevelProbeArgs a;
  a.sync = (unsigned int *)d_ws;
  a.pairs = (char *)d_ws + kProbePairsOffset;
  a.status = d_status;
  a.levels = levels;
  a.mode = mode;
  // tags tag0 .. tag0 + levels - 1 are this launch's own; 0 is never used
  uint32_t t0 = g_probe_tag.fetch_add((uint32_t)levels + 1u) + 1u;
  if (t0 == 0 || t0 + (uint32_t)levels < t0) t0 = g_probe_tag.fetch_add((uint32_t)levels + 1u) + 1u;
  a.tag0 = t0;
  a.timeout = barrier_timeout_ticks();
  return launch_persistent(probe_levels_kernel, grid, kProbeThreads, 0, a, stream);
}

extern "C" size_t cortex_probe_mfma_sink_floats(void) {
  const int cus = num_cus();
  return cus > 0 ? (size_t)cus * 64 * kProbeWaves : 0;
}

extern "C" double cortex_probe_mfma_flops(int32_t iters) {
  const int cus = num_cus();
  if (cus <= 0 || iters < 0) return 0.0;
  return (double)cus * kProbeWaves * iters * kProbeChains * kProbeSteps * (16.0 * 16.0 * 4.0 * 2.0);
}

extern "C" int cortex_probe_mfma(float *d_sink, int32_t iters, void *stream) {
  const int cus = num_cus();
  if (!d_sink || iters < 0) return CORTEX_E_INVAL;
  if (cus <= 0) return CORTEX_E_HIP;
  hipLaunchKernelGGL(probe_mfma_kernel, dim3(cus), dim3(64 * kProbeWaves), 0, (hipStream_t)stream, d_sink, iters, 1.0f);
  return hipGetLastError() == hipSuccess ? CORTEX_OK : CORTEX_E_HIP;
}
