// Diagnostics: a throughput probe of the fp32 matrix cores, so that achieved
// rates can be set against what the chip sustains, beside its nominal peak.
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

}  // namespace cortex

using namespace cortex;

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
