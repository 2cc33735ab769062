// Library-wide host state: launch knobs, the grids of the last launches and
// the version string.
#include <atomic>
#include <map>
#include <mutex>

#include "cortex_host.hpp"

namespace cortex {

constexpr int kKnobs = 8;
// The default spin limit of one wait, 0.2 s, is about 10^4 times the longest
// level or linearizer phase measured on the largest batch here (tens of
// microseconds): a wait that long means the grid is not co-resident (a GPU
// shared with other persistent work), and the launch then ends with a status
// instead of holding the GPU.
static std::atomic<int64_t> g_knobs[kKnobs] = {{0}, {0}, {200000}, {0}, {0}, {0}, {0}, {0}};
static std::atomic<int32_t> g_last_grid[2] = {{0}, {0}};

int64_t knob(int32_t which) {
  if (which < 0 || which >= kKnobs) return 0;
  return g_knobs[which].load();
}

// Per-device CU counts and per-kernel occupancies, queried once.
constexpr int kMaxDevices = 64;
static std::atomic<int> g_cus[kMaxDevices];
static std::mutex g_occ_mu;
static std::map<std::pair<const void *, long long>, int> g_occ;

int num_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  int c = g_cus[dev].load();
  if (c > 0) return c;
  if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  g_cus[dev].store(c);
  return c;
}

int cached_occupancy(const void *kernel, int threads, size_t dyn_lds) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  std::lock_guard<std::mutex> lock(g_occ_mu);
  auto key = std::make_pair(kernel, ((long long)dev << 40) | ((long long)threads << 24) | (long long)dyn_lds);
  auto it = g_occ.find(key);
  if (it != g_occ.end()) return it->second;
  int per_cu = 0;
  // A request beyond the compute unit's LDS fails here: report no occupancy
  // and clear the runtime's last error, which would otherwise surface at the
  // caller's next HIP call.
  if (dyn_lds > 0 &&
      hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds) != hipSuccess) {
    (void)hipGetLastError();
    g_occ[key] = 0;
    return 0;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, dyn_lds) != hipSuccess) {
    (void)hipGetLastError();
    return -1;
  }
  g_occ[key] = per_cu;
  return per_cu;
}

void set_last_grid(int which, int32_t grid) {
  if (which >= 0 && which < 2) g_last_grid[which].store(grid);
}

}  // namespace cortex

extern "C" int cortex_set_knob(int32_t which, int64_t value) {
  if (which < 0 || which >= cortex::kKnobs || value < 0) return CORTEX_E_INVAL;
  if (which == CORTEX_KNOB_LEVEL_SYNC && value > 3) return CORTEX_E_INVAL;
  if (which == CORTEX_KNOB_TREE_UNROLL && value > 2) return CORTEX_E_INVAL;
  if (which == CORTEX_KNOB_ABLATE && value > 7) return CORTEX_E_INVAL;
  cortex::g_knobs[which].store(value);
  return CORTEX_OK;
}

extern "C" int64_t cortex_get_knob(int32_t which) { return cortex::knob(which); }

extern "C" int32_t cortex_last_grid(int32_t which) {
  if (which < 0 || which > 1) return 0;
  return cortex::g_last_grid[which].load();
}

extern "C" const char *cortex_version(void) { return "cortex-mi355x 0.1 (gfx950)"; }
