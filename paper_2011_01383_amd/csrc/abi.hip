// Library-wide host state: launch knobs, the grids of the last launches and
// the version string.
#include <atomic>

#include "cortex_host.hpp"

namespace cortex {

static std::atomic<int64_t> g_knobs[3] = {{0}, {0}, {5000000}};
static std::atomic<int32_t> g_last_grid[2] = {{0}, {0}};

int64_t knob(int32_t which) {
  if (which < 0 || which > 2) return 0;
  return g_knobs[which].load();
}

void set_last_grid(int which, int32_t grid) {
  if (which >= 0 && which < 2) g_last_grid[which].store(grid);
}

}  // namespace cortex

extern "C" int cortex_set_knob(int32_t which, int64_t value) {
  if (which < 0 || which > 2 || value < 0) return CORTEX_E_INVAL;
  cortex::g_knobs[which].store(value);
  return CORTEX_OK;
}

extern "C" int64_t cortex_get_knob(int32_t which) { return cortex::knob(which); }

extern "C" int32_t cortex_last_grid(int32_t which) {
  if (which < 0 || which > 1) return 0;
  return cortex::g_last_grid[which].load();
}

extern "C" const char *cortex_version(void) { return "cortex-mi355x 0.1 (gfx950)"; }
