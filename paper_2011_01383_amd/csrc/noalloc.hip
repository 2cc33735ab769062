// cortex_tree_infer_noalloc: the whole path of a tree batch (the call
// cortex_tree_infer makes) for callers that cannot allocate device memory,
// with the workspace in a library-owned array instead of a caller's buffer.
//
// The array, `scratch`, is a file-scope device array of kScratchBytes.  Each
// GPU the library runs on holds its own copy until the process ends.  Host
// code never passes the array's name to a kernel or a copy: at the first call
// on a device, with that device current, hipGetSymbolAddress gives the copy's
// device address, which is kept per device and used from then on.
//
// The array is cut into regions at fixed offsets, whatever the batch, so each
// region only ever holds its own kind of data:
//   [0, 256)          preparation header: a 64-bit marker of a cleared array
//   forward header    barrier words, the staging epoch, entered words (and the
//                     trace area in trace builds)
//   linearizer        the workspace of cortex_linearize (two-launch batches)
//   h staging         tagged (value, tag) pairs of h
//   second staging    tagged pairs of c, P or the TreeGRU reset sums
//   phase values      the TreeGRU values kept across a barrier (LEVEL_SYNC 3)
// The staging regions hold nothing but pairs written under the forward
// header's epoch, so every tag in them is at most the epoch and a launch's tag
// (the epoch plus one) is never found there before the launch writes it.
//
// Every call first enqueues noalloc_prepare_kernel (one workgroup): it clears
// both headers' barrier words and advances the staging epoch, so a call that
// follows one that failed (its barrier words may be left ahead, its epoch not
// advanced) needs no reset.  The first time on a device (no marker yet), or
// when the epoch nears its end, it clears the whole array instead.  Calls on
// one GPU share its array and therefore must not overlap in time.
#include <mutex>

#include "cortex_device.hpp"
#include "cortex_host.hpp"

namespace cortex {

constexpr size_t kScratchBytes = CORTEX_NOALLOC_SCRATCH_BYTES;
constexpr size_t kPrepBytes = 256;
constexpr size_t kLinCap = 2u << 20;       // linearizer workspace
constexpr size_t kHsCap = 16u << 20;       // h staging: N * H <= 2,097,152
constexpr size_t kCsCap = 32u << 20;       // c / P / reset-sum staging: 4,194,304 pairs
constexpr size_t kKeepCap = 8u << 20;      // TreeGRU phase values: N * H * 3 floats
constexpr unsigned long long kClearedMarker = 0x5343524154434832ull;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchMap {
  size_t fwd, lin, hs, cs, keep, end;
};

static ScratchMap scratch_map() {
  ScratchMap m;
  m.fwd = kPrepBytes;
  m.lin = m.fwd + align_up(forward_header_bytes(), 256);
  m.hs = m.lin + kLinCap;
  m.cs = m.hs + kHsCap;
  m.keep = m.cs + kCsCap;
  m.end = m.keep + kKeepCap;
  return m;
}

// One workgroup.  base is the device address of this GPU's array.
__global__ void __launch_bounds__(1024) noalloc_prepare_kernel(unsigned char *base, unsigned long long total,
                                                               unsigned int fwd_off, unsigned int lin_off) {
  unsigned long long *marker = (unsigned long long *)base;
  unsigned int *fwd = (unsigned int *)(base + fwd_off);
  unsigned int *lin = (unsigned int *)(base + lin_off);
  __shared__ int s_full;
  __shared__ unsigned int s_epoch;
  if (threadIdx.x == 0) {
    const unsigned int e = fwd[kEpochWord];
    s_full = *marker != kClearedMarker || e >= 0xFFFFFF00u;
    s_epoch = e;
  }
  __syncthreads();
  if (s_full) {
    // the whole array (the marker's own bytes are cleared by thread 0 before
    // it writes the marker)
    const uint4 z = make_uint4(0u, 0u, 0u, 0u);
    for (unsigned long long i = (unsigned long long)threadIdx.x * 16u; i < total;
         i += (unsigned long long)blockDim.x * 16u)
      *(uint4 *)(base + i) = z;
    if (threadIdx.x == 0) *marker = kClearedMarker;
    return;
  }
  // barrier and entered words of both headers; the forward's epoch advances
  // by one, past the tag of a launch that may have stopped on an error
  for (unsigned int i = threadIdx.x; i < (unsigned int)(kSyncBytes / 4); i += blockDim.x) {
    if (i != (unsigned int)kEpochWord) fwd[i] = 0u;
    lin[i] = 0u;
  }
  if (threadIdx.x == 0) fwd[kEpochWord] = s_epoch + 1u;
}

constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static unsigned char *g_scratch[kMaxScratchDevices];

// This device's copy of the array (looked up once per device).
static unsigned char *device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch[dev] = (unsigned char *)p;
  }
  return g_scratch[dev];
}

}  // namespace cortex

using namespace cortex;

extern "C" int cortex_tree_infer_noalloc(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                                         const float *d_x_table, int32_t x_rows, const int32_t *d_x_index,
                                         const float *d_leaf_mat, const cortex_weights_t *w, float *d_h,
                                         float *d_c_or_P, int32_t *d_status, void *stream) {
  if (!lin || !w || !d_status || x_rows < 0 || !lin->height || !lin->node_row) return CORTEX_E_INVAL;
  if (cell < CORTEX_TREE_RNN || cell > CORTEX_SIMPLE_TREEGRU) return CORTEX_E_INVAL;
  const int32_t N = lin->num_nodes, K = lin->max_arity;
  if (N < 0 || K < 1 || K > 4) return CORTEX_E_INVAL;
  const ScratchMap m = scratch_map();
  if (m.end > kScratchBytes) return CORTEX_E_INVAL;       // a build whose header outgrew the array
  unsigned char *base = device_scratch();
  if (!base) return CORTEX_E_HIP;
  FwdRegions reg;
  if (N > 0) {
    if (cortex_tree_infer_workspace_bytes(cell, N, K, H) == 0) return CORTEX_E_INVAL;
    if (align_up(cortex_linearize_workspace_bytes(N, K), 256) > kLinCap) return CORTEX_E_WORKSPACE;
    if (!fixed_regions(cell, N, H, base + m.fwd, m.lin - m.fwd, base + m.hs, kHsCap, base + m.cs, kCsCap,
                       base + m.keep, kKeepCap, reg))
      return CORTEX_E_WORKSPACE;
  } else {
    reg = FwdRegions{base + m.fwd, nullptr, nullptr, nullptr};
  }
  // every host check first, so a call that returns an error enqueues nothing
  int rc = tree_infer_impl(cell, H, d_children, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P,
                           d_status, base + m.lin, kLinCap, base + m.fwd, m.end - m.fwd, &reg, stream, true);
  if (rc != CORTEX_OK) return rc;
  unsigned char *b = base;
  unsigned long long total = (unsigned long long)m.end;
  unsigned int fwd_off = (unsigned int)m.fwd, lin_off = (unsigned int)m.lin;
  void *kargs[] = {(void *)&b, (void *)&total, (void *)&fwd_off, (void *)&lin_off};
  if (hipLaunchKernel((const void *)noalloc_prepare_kernel, dim3(1), dim3(1024), kargs, 0, (hipStream_t)stream) !=
      hipSuccess)
    return CORTEX_E_HIP;
  return tree_infer_impl(cell, H, d_children, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P,
                         d_status, base + m.lin, kLinCap, base + m.fwd, m.end - m.fwd, &reg, stream, false);
}
