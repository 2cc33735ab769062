// Persistent level-synchronous forward kernels (Sec. 4.1 loop nest; kernel
// fusion and model persistence as evaluated in Sec. 7.2-7.3).
//
// One launch runs every level.  Workgroup b owns hidden slice s = b / Q
// (J hidden units, all gates of those units) and node group q = b % Q (the
// TreeGRU kernel: s = b % S, q = b / S).  Its
// slice of the cell weights is loaded into LDS once and stays there for the
// whole pass (persistence).  The rows of level l are cut into 16-row tiles
// starting at the level's first row; group q takes the tiles u with
// (u + l) % Q == q.  For a tile, each of the 8 waves loads its share of the
// operand rows (child states, and the node input where the cell fuses it)
// straight into registers in the MFMA operand layout and contracts it with the
// resident weight slice on the fp32 MFMA units; the partial sums meet in LDS,
// where the threads of the workgroup apply the gate nonlinearities together
// and write the slice's J columns of the new states.
//
// Levels are ordered per datum, not by a device-wide barrier.  The dependence
// is carried by the level loop (Appendix A.4) and a level only reads lower
// levels, so it suffices that every state element is also published as a
// (value, launch tag) pair with one device-scope store and that a consumer
// waits for exactly the elements it reads.  TreeRNN and N-ary TreeLSTM leaves
// are the inputs themselves (specialization, Sec. 3.1; zero initial memory
// cell, Sec. 4.3): a level reading a leaf child takes the row from the input
// table directly, so nothing ever waits on the leaf level.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "cortex_device.hpp"
#include "cortex_host.hpp"
#include "lin_small.hpp"

namespace cortex {

constexpr int kFwdThreads = 512;
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kTileM = 16;
constexpr int CELL_DAG = 16;                 // internal id of the DAG-RNN cell

// Optional timeline (builds with -DCORTEX_TRACE only): every workgroup (up to
// kTraceBlocks) stamps the 100 MHz wall clock at phase boundaries of every
// level into trace[block][kTraceLevels][16] (uint64), placed in the workspace
// after the barrier words: slots 0-5 are phases seen by wave 0, slot 8 + w is
// the time wave w had all its operands.  Row kTraceLevels-1 holds kernel-wide
// stamps: entry, weights loaded, structure ready, exit.
constexpr int kTraceLevels = 64;
constexpr int kTraceBlocks = 256;
constexpr int kTraceSlots = 16;
#ifdef CORTEX_TRACE
constexpr size_t kTraceBytes = (size_t)kTraceBlocks * kTraceLevels * kTraceSlots * sizeof(uint64_t);
#define CORTEX_TRACE_AT(row, k)                                                                        \
  do {                                                                                                \
    if (threadIdx.x == 0 && blockIdx.x < kTraceBlocks)                                                \
      a.trace[((size_t)blockIdx.x * kTraceLevels + (row)) * kTraceSlots + (k)] = wall_clock64();      \
  } while (0)
#define CORTEX_TRACE_POINT(lvl, k) CORTEX_TRACE_AT(min((lvl), kTraceLevels - 2), k)
#define CORTEX_TRACE_KERNEL(k) CORTEX_TRACE_AT(kTraceLevels - 1, k)
#define CORTEX_TRACE_WAVE(lvl)                                                                          \
  do {                                                                                                \
    if ((threadIdx.x & 63) == 0 && blockIdx.x < kTraceBlocks)                                         \
      a.trace[((size_t)blockIdx.x * kTraceLevels + min((lvl), kTraceLevels - 2)) * kTraceSlots + 8 +   \
              (threadIdx.x >> 6)] = wall_clock64();                                                   \
  } while (0)
#else
constexpr size_t kTraceBytes = 0;
#define CORTEX_TRACE_POINT(lvl, k) \
  do {                             \
  } while (0)
#define CORTEX_TRACE_KERNEL(k) \
  do {                         \
  } while (0)
#define CORTEX_TRACE_WAVE(lvl) \
  do {                         \
  } while (0)
#endif

struct FwdArgs {
  int32_t N, K, S, Q, x_rows;
  const int32_t *num_levels, *level_offsets, *level_nodes, *child_rows;
  const float *x_table;
  const int32_t *x_index;
  const float *leaf_mat;
  const float *x;
  const float *W, *U, *b, *W_M;
  float *h, *c;
  int32_t *status;
  unsigned int *sync;
  uint64_t timeout;
  uint64_t *trace;
  int32_t retire;               // 1: publish this launch's tag as the workspace's staging epoch at the end
                                // (0 for all but the last of a sequence of per-level launches)
  void *hs, *cs;                // tagged staging of h and c (workspace)
  int32_t level_lo, level_hi;   // levels this launch runs (all of them unless one launch per level)
  int32_t level_barrier;        // 1: a device-wide barrier closes every level (instead of per-datum waits alone);
                                // 2 (TreeGRU): also one between the level's two exchanges
  float *keep;                  // TreeGRU, level_barrier 2: z, W_h x + b_h and h~ per (row, unit), [3][N][H]
  // fused launch (cortex_tree_infer): the children to linearize, and where
  // workgroup 0 writes the linearization
  const int32_t *children;
  int32_t *o_num_levels, *o_height, *o_level_offsets, *o_level_nodes, *o_node_row, *o_child_rows;
  int32_t ablate;               // slice kernel, for ablation studies: bit 0 (its own instance) reads the weight slice from
                                // memory at every tile instead of LDS; bit 1 stages the leaf states and
                                // has parents wait for them instead of reading their inputs directly
  float *pre;                   // DAG-RNN with hoisted input products: W x + b of every row, [N][H] in row order
};

// ---------------------------------------------------------------------------
// Level structure: the linearization, cached in LDS when it fits.
//   off[L+1]  level offsets;  crow[N*K]  child rows;  xrow[N]  input row of
//   each row (x_index of its node; -1 = none) for the cells that read inputs
//   through rows;  node[N]  node id of each row (DAG-RNN input).
// ---------------------------------------------------------------------------
template <bool kCached>
struct Structure {
  const int *off, *crow, *xrow, *node;
  int K;
  __device__ int offset(int l) const { return off[l]; }
  __device__ int child(int r, int s) const { return crow[r * K + s]; }
  __device__ int input_row(int r) const { return xrow[r]; }
  __device__ int node_of(int r) const { return node[r]; }
};

// Gates, contraction depth and default units per slice of each cell.
template <int CELL, int H>
struct Cell;
template <int H>
struct Cell<CORTEX_TREE_RNN, H> {
  static constexpr int GATES = 1, KA = 2 * H, J = (H <= 64) ? H : 16;
};
template <int H>
struct Cell<CORTEX_NARY_TREELSTM, H> {
  static constexpr int GATES = 5, KA = 2 * H, J = 4;
};
template <int H>
struct Cell<CORTEX_CHILDSUM_TREELSTM, H> {
  static constexpr int GATES = 4, KA = 2 * H, J = 4;
};
template <int H>
struct Cell<CELL_DAG, H> {
  static constexpr int GATES = 1, KA = 3 * H, J = 16;
};

template <int CELL, int H, int J_>
struct Dims {
  static constexpr int J = J_, GATES = Cell<CELL, H>::GATES, KA = Cell<CELL, H>::KA;
  static constexpr int GJ = GATES * J;                     // weight-slice rows
  static constexpr int MPAD = (GJ + 15) / 16 * 16;
  static constexpr int NT = MPAD / 16;
  static constexpr bool kChildSum = CELL == CORTEX_CHILDSUM_TREELSTM;
  // k range per wave, padded to whole 16-blocks (zeros beyond KA)
  static constexpr int KW = ((KA + kFwdWaves * 16 - 1) / (kFwdWaves * 16)) * 16;
  static constexpr int NB = KW / 16;                       // float4 operand loads per lane per tile
  // child-sum: node part over 4 waves, edge part (64 edge rows) in two k halves
  static constexpr int KWX = H / 4, NBX = KWX / 16;
  static constexpr int KWE = H / 2, NBE = KWE / 16;
  static constexpr int LDW = kChildSum ? (2 * H + 4) : (kFwdWaves * KW + 4);   // weight row stride
  static_assert(H % J == 0, "slices must tile H");
  static_assert(H % 64 == 0, "H must be a multiple of 64");
};

// Weight-slice row m = (gate g, unit j); child-sum rows are ordered
// (i, o, u, f) while the input layout is (i, f, o, u).
__device__ __forceinline__ int childsum_gate(int gslot) {
  return gslot == 0 ? 0 : (gslot == 1 ? 2 : (gslot == 2 ? 3 : 1));
}

// The workgroup's weight slice, copied into LDS: issue_weight_slice requests
// every value of the thread (registers), commit_weight_slice stores them, so
// the copy costs about one memory round trip, which other loads issued
// between the two calls share.
template <int CELL, int H, int J>
struct WeightRegs {
  using D = Dims<CELL, H, J>;
  static constexpr int ROW4 = (D::LDW - 4) / 4, ITEMS = D::MPAD * ROW4;
  static constexpr int PER = (ITEMS + kFwdThreads - 1) / kFwdThreads;
  float4 v[PER];
  float bv;                       // bias of slice row threadIdx.x (< MPAD)
};

template <int CELL, int H, int J>
__device__ __forceinline__ void issue_weight_slice(const FwdArgs &a, int hbase, WeightRegs<CELL, H, J> &w) {
  using D = Dims<CELL, H, J>;
  using WR = WeightRegs<CELL, H, J>;
  constexpr int ROW4 = WR::ROW4, SEG4 = H / 4, KA4 = D::KA / 4, ITEMS = WR::ITEMS;
  static_assert(D::MPAD <= kFwdThreads, "one bias per thread");
#pragma unroll
  for (int k = 0; k < WR::PER; ++k) {
    const int idx = threadIdx.x + k * kFwdThreads;
    const int m = idx / ROW4, c4 = idx % ROW4;
    const int g = m / J, j = m % J, hj = hbase + j;
    const int sg = c4 / SEG4, o4 = c4 % SEG4;
    w.v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (idx < ITEMS && m < D::GJ && c4 < KA4) {
      const float *src = nullptr;
      if (CELL == CORTEX_TREE_RNN) src = a.W + (size_t)hj * 2 * H + sg * H;
      if (CELL == CORTEX_NARY_TREELSTM) src = a.U + ((size_t)(sg * 5 + g) * H + hj) * H;
      if (CELL == CORTEX_CHILDSUM_TREELSTM)
        src = (sg == 0 ? a.W : a.U) + ((size_t)childsum_gate(g) * H + hj) * H;
      if (CELL == CELL_DAG) src = (sg == 0 ? a.W : a.U + (size_t)(sg - 1) * H * H) + (size_t)hj * H;
      w.v[k] = *(const float4 *)(src + o4 * 4);
    }
  }
  const int m = threadIdx.x;
  w.bv = 0.f;
  if (m < D::GJ) {
    const int g = m / J, hj = hbase + m % J;
    if (CELL == CORTEX_TREE_RNN || CELL == CELL_DAG) w.bv = a.b[hj];
    if (CELL == CORTEX_NARY_TREELSTM) w.bv = a.b[g * H + hj];
    if (CELL == CORTEX_CHILDSUM_TREELSTM) w.bv = a.b[childsum_gate(g) * H + hj];
  }
}

template <int CELL, int H, int J>
__device__ __forceinline__ void commit_weight_slice(const WeightRegs<CELL, H, J> &w, float *W_s, float *bias_s) {
  using D = Dims<CELL, H, J>;
  using WR = WeightRegs<CELL, H, J>;
#pragma unroll
  for (int k = 0; k < WR::PER; ++k) {
    const int idx = threadIdx.x + k * kFwdThreads;
    if (idx < WR::ITEMS) *(float4 *)&W_s[(idx / WR::ROW4) * D::LDW + (idx % WR::ROW4) * 4] = w.v[k];
  }
  if (threadIdx.x < D::MPAD) bias_s[threadIdx.x] = w.bv;
}

template <int CELL, int H, int J>
__device__ void load_weight_slice(const FwdArgs &a, int hbase, float *W_s, float *bias_s) {
  WeightRegs<CELL, H, J> w;
  issue_weight_slice<CELL, H, J>(a, hbase, w);
  commit_weight_slice<CELL, H, J>(w, W_s, bias_s);
}

// Four consecutive columns c .. c+3 of weight-slice row m (the values
// load_weight_slice places in LDS), read from the weight tensors.
template <int CELL, int H, int J>
__device__ __forceinline__ float4 weight_slice_at(const FwdArgs &a, int hbase, int m, int c) {
  using D = Dims<CELL, H, J>;
  if (m >= D::GJ || c >= D::KA) return make_float4(0.f, 0.f, 0.f, 0.f);
  const int g = m / J, hj = hbase + m % J, sg = c / H, o = c % H;
  const float *src = nullptr;
  if (CELL == CORTEX_TREE_RNN) src = a.W + (size_t)hj * 2 * H + sg * H;
  if (CELL == CORTEX_NARY_TREELSTM) src = a.U + ((size_t)(sg * 5 + g) * H + hj) * H;
  if (CELL == CORTEX_CHILDSUM_TREELSTM) src = (sg == 0 ? a.W : a.U) + ((size_t)childsum_gate(g) * H + hj) * H;
  if (CELL == CELL_DAG) src = (sg == 0 ? a.W : a.U + (size_t)(sg - 1) * H * H) + (size_t)hj * H;
  return *(const float4 *)(src + o);
}

// Fills the structure cache in LDS (kCached) or points at global memory.
// Validates what the level loop relies on: 1 <= L <= N, monotone offsets
// ending at N, child rows in a strictly lower level, input rows in range.
template <bool kCached, bool kNeedX, bool kNeedNode>
__device__ bool setup_structure(const FwdArgs &a, int *cache, Structure<kCached> &st, int &L) {
  L = *a.num_levels;
  const int N = a.N, K = a.K;
  if (L < 1 || L > N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return false;
  }
  st.K = K;
  if (kCached) {
    int *off = cache, *crow = cache + (L + 1), *xrow = crow + N * K, *node = xrow + (kNeedX ? N : 0);
    for (int i = threadIdx.x; i <= L; i += kFwdThreads) off[i] = a.level_offsets[i];
    for (int i = threadIdx.x; i < N * K; i += kFwdThreads) crow[i] = a.child_rows[i];
    for (int r = threadIdx.x; r < N; r += kFwdThreads) {
      int v = a.level_nodes[r];
      if (v < 0 || v >= N) { raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION); v = -1; }
      if (kNeedNode) node[r] = v;
      if (kNeedX) {
        int xi = v >= 0 ? a.x_index[v] : -1;
        if (xi < -1 || xi >= a.x_rows) { raise_status(a.status, CORTEX_ST_INPUT_RANGE); xi = -1; }
        xrow[r] = xi;
      }
    }
    st.off = off;
    st.crow = crow;
    st.xrow = xrow;
    st.node = node;
  } else {
    st.off = a.level_offsets;
    st.crow = a.child_rows;
    st.xrow = nullptr;
    st.node = a.level_nodes;
  }
  __syncthreads();
  // offsets: 0 = off[0] <= ... <= off[L] = N
  int bad = 0;
  for (int l = threadIdx.x; l < L; l += kFwdThreads) {
    const int o0 = st.offset(l), o1 = st.offset(l + 1);
    if (o1 < o0 || (l == 0 && o0 != 0) || (l == L - 1 && o1 != N)) bad = 1;
  }
  // every child row lies in a strictly lower level than its parent row; the
  // level of a row is found by binary search over the offsets
  for (int r = threadIdx.x; r < N && !bad; r += kFwdThreads) {
    int lo = 0, hi = L - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (st.offset(mid) <= r) lo = mid;
      else hi = mid - 1;
    }
    const int start = st.offset(lo);
    for (int s = 0; s < K; ++s) {
      const int cr = st.child(r, s);
      if (cr < -1 || cr >= start) bad = 1;
    }
  }
  if (__syncthreads_or(bad)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return false;
  }
  return true;
}

// Child rows and input rows of up to kChunkTiles of a workgroup's tiles in one
// level (child-sum kernel), staged into LDS in one pass when the whole
// linearization is not cached: operand addresses then never wait on a global
// load.  Chunk tile k is level tile u0 + k*Q, rows r0 + 16*(u0 + k*Q) + i.
constexpr int kChunkTiles = 16;
struct ChunkRows {
  int crow[kChunkTiles][kTileM][4];     // child rows, -1 = none
  int xrow[kChunkTiles][kTileM];
};

__device__ void stage_chunk(const FwdArgs &a, ChunkRows &cr, int u0, int ntiles, int Q, int r0, int r1) {
  for (int idx = threadIdx.x; idx < ntiles * kTileM; idx += kFwdThreads) {
    const int k = idx / kTileM, i = idx % kTileM;
    const int row = r0 + (u0 + k * Q) * kTileM + i;
    const bool live = row < r1;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      int c = (live && s < a.K) ? a.child_rows[(size_t)row * a.K + s] : -1;
      if (c < -1 || c >= r0) {                    // a child must sit in a lower level
        raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
        c = -1;
      }
      cr.crow[k][i][s] = c;
    }
    int v = live ? a.level_nodes[row] : -1;
    if (v < -1 || v >= a.N) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      v = -1;
    }
    int xi = v >= 0 ? a.x_index[v] : -1;
    if (xi < -1 || xi >= a.x_rows) {
      raise_status(a.status, CORTEX_ST_INPUT_RANGE);
      xi = -1;
    }
    cr.xrow[k][i] = xi;
  }
}

// ---------------------------------------------------------------------------
// Operand sources of the slice kernels.  A row of the contraction operand is
// SEGS segments of H values (the two child slots; for DAG-RNN the node input,
// then the two child slots).  Each (row, segment) gets one code:
//   c >= 0    the staged state of row c (a child computed in this launch)
//   c <= -2   plain row -2-c: the input-table row of a leaf child (TreeRNN,
//             N-ary TreeLSTM, whose leaves are their inputs) or the node's own
//             input row (DAG-RNN, segment 0)
//   -1        no source: the segment reads zeros
// so that forming a tile's load addresses takes one LDS read per segment.
// ---------------------------------------------------------------------------
template <int CELL>
struct SrcCfg {
  static constexpr int SEGS = CELL == CELL_DAG ? 3 : 2;
  static constexpr bool kLeafX = CELL == CORTEX_TREE_RNN || CELL == CORTEX_NARY_TREELSTM;
  static constexpr bool kDag = CELL == CELL_DAG;
};
// Largest N whose codes are kept in LDS (the host checks the same bound).
constexpr int kMaxCachedRows = 2560;
constexpr int kCachedRowsPerThread = (kMaxCachedRows + kFwdThreads - 1) / kFwdThreads;

// Cached: off[L+1], codes[N*SEGS] and (leaf-input cells) the input row of
// every row, xrow[N], all in LDS.  Uncached: offsets from global memory and
// codes staged per chunk of tiles.  Validates 1 <= L <= N, monotone offsets
// from 0 to N, child rows in a strictly lower level, node ids and input rows
// in range.
//
// The cached path is split in two: prefetch_sources requests every value it
// needs (the level count, all N + 1 entries of the offsets array, whose
// capacity is N + 1, the node ids and child rows of every row, and the input
// row of every node id) into registers, with no load depending on another,
// so they share one memory round trip, also with the weight loads issued
// beside them; setup_sources then builds the cache from the registers (the
// input row of a row is gathered through LDS).
struct SrcRegs {
  int L;
  int ch[kCachedRowsPerThread][2];
  int node[kCachedRowsPerThread];
  int xi[kCachedRowsPerThread];          // x_index of node id tid + k*threads
  int off[kCachedRowsPerThread + 1];     // level_offsets[tid + k*threads]
};

template <int CELL, bool kCached>
__device__ __forceinline__ void prefetch_sources(const FwdArgs &a, SrcRegs &p) {
  using SC = SrcCfg<CELL>;
  const int N = a.N, K = a.K, tid = threadIdx.x;
  p.L = *a.num_levels;
  if (!kCached) return;
#pragma unroll
  for (int k = 0; k < kCachedRowsPerThread; ++k) {
    const int r = tid + k * kFwdThreads;
#pragma unroll
    for (int s = 0; s < 2; ++s) p.ch[k][s] = (r < N && s < K) ? a.child_rows[r * K + s] : -1;
    p.node[k] = r < N ? a.level_nodes[r] : -1;
    p.xi[k] = (SC::kLeafX && r < N) ? a.x_index[r] : -1;
  }
#pragma unroll
  for (int k = 0; k <= kCachedRowsPerThread; ++k) {
    const int i = tid + k * kFwdThreads;
    p.off[k] = i <= N ? a.level_offsets[i] : 0;
  }
}

template <int CELL, bool kCached>
__device__ bool setup_sources(const FwdArgs &a, const SrcRegs &p, int *cache, int &L, const int *&off,
                              const int *&codes, const int *&xrow) {
  using SC = SrcCfg<CELL>;
  constexpr int SEGS = SC::SEGS;
  const int N = a.N, K = a.K;
  const int tid = threadIdx.x;
  L = p.L;
  if (L < 1 || L > N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return false;
  }
  int bad = 0;
  if (!kCached) {
    off = a.level_offsets;
    codes = nullptr;
    xrow = nullptr;
    for (int l = tid; l < L; l += kFwdThreads) {
      const int o0 = off[l], o1 = off[l + 1];
      if (o1 < o0 || (l == 0 && o0 != 0) || (l == L - 1 && o1 != N)) bad = 1;
    }
    if (__syncthreads_or(bad)) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return false;
    }
    return true;
  }
  int *o = cache, *cd = cache + (L + 1), *xr = cd + N * SEGS;
  int *xnode = cd;                 // input row by node id, until the codes are written (N <= N*SEGS ints)
#pragma unroll
  for (int k = 0; k <= kCachedRowsPerThread; ++k) {
    const int i = tid + k * kFwdThreads;
    if (i <= L) o[i] = p.off[k];
  }
#pragma unroll
  for (int k = 0; k < kCachedRowsPerThread; ++k) {
    const int r = tid + k * kFwdThreads;
    if (r >= N) break;
    const int v = p.node[k];
    if (v < 0 || v >= N) bad = 1;
    if (SC::kLeafX) {
      int xi = p.xi[k];
      if (xi < -1 || xi >= a.x_rows) {
        raise_status(a.status, CORTEX_ST_INPUT_RANGE);
        xi = -1;
      }
      xnode[r] = xi;
    }
  }
  if (SC::kLeafX) __syncthreads();
#pragma unroll
  for (int k = 0; k < kCachedRowsPerThread; ++k) {
    const int r = tid + k * kFwdThreads;
    if (r >= N) break;
    const int v = p.node[k];
    const bool vok = v >= 0 && v < N;
    if (SC::kLeafX) xr[r] = vok ? xnode[v] : -1;
    if (SC::kDag) cd[r * SEGS] = vok ? -2 - v : -1;
  }
  __syncthreads();                 // offsets and input rows complete; xnode no longer read
  for (int l = tid; l < L; l += kFwdThreads) {
    const int o0 = o[l], o1 = o[l + 1];
    if (o1 < o0 || (l == 0 && o0 != 0) || (l == L - 1 && o1 != N)) bad = 1;
  }
  const int off1 = o[1];
#pragma unroll
  for (int k = 0; k < kCachedRowsPerThread; ++k) {
    const int r = tid + k * kFwdThreads;
    if (r >= N) break;
    // the level of row r, by binary search over the offsets
    int lo = 0, hi = L - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (o[mid] <= r) lo = mid;
      else hi = mid - 1;
    }
    const int start = o[lo];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      int c = p.ch[k][s];
      if (c < -1 || c >= start) {          // a child must sit in a strictly lower level
        bad = 1;
        c = -1;
      }
      if (SC::kLeafX && !(a.ablate & 2) && c >= 0 && c < off1) c = xr[c] >= 0 ? -2 - xr[c] : -1;
      if (s < K) cd[r * SEGS + (SC::kDag ? s + 1 : s)] = c;
    }
  }
  if (__syncthreads_or(bad)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return false;
  }
  off = o;
  codes = cd;
  xrow = xr;
  return true;
}

// Codes of up to kChunkTiles of a workgroup's tiles in one level (uncached
// linearization), staged into LDS in one pass.  Chunk tile k is level tile
// u0 + k*Q, rows r0 + 16*(u0 + k*Q) + i.
struct ChunkSrc {
  int code[kChunkTiles][kTileM][3];
};

template <int CELL>
__device__ void stage_chunk_codes(const FwdArgs &a, ChunkSrc &cs, int u0, int ntiles, int Q, int r0, int r1,
                                  int off1) {
  using SC = SrcCfg<CELL>;
  for (int idx = threadIdx.x; idx < ntiles * kTileM; idx += kFwdThreads) {
    const int k = idx / kTileM, i = idx % kTileM;
    const int row = r0 + (u0 + k * Q) * kTileM + i;
    const bool live = row < r1;
    if (SC::kDag) {
      const int v = live ? a.level_nodes[row] : -1;
      if (v < -1 || v >= a.N) raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      cs.code[k][i][0] = (v >= 0 && v < a.N) ? -2 - v : -1;
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      int c = (live && s < a.K) ? a.child_rows[(size_t)row * a.K + s] : -1;
      if (c < -1 || c >= r0) {                    // a child must sit in a lower level
        raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
        c = -1;
      }
      if (SC::kLeafX && !(a.ablate & 2) && c >= 0 && c < off1) {     // a leaf child: its input row
        const int v = a.level_nodes[c];
        int xi = -1;
        if (v < 0 || v >= a.N) raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
        else xi = a.x_index[v];
        if (xi < -1 || xi >= a.x_rows) {
          raise_status(a.status, CORTEX_ST_INPUT_RANGE);
          xi = -1;
        }
        c = xi >= 0 ? -2 - xi : -1;
      }
      cs.code[k][i][SC::kDag ? s + 1 : s] = c;
    }
  }
}

// Leaf level of TreeRNN / N-ary TreeLSTM, spread over every thread of the
// launch: h = input row (or 0), c = 0.  Nothing waits on these rows (parents
// read leaf children from the input table), so they are not staged, except
// under ablation bit 1, where parents wait for them like any other child.
template <int H, bool kWithC>
__device__ void write_leaf_outputs(const FwdArgs &a, const int *xrow, int r1, const TagBuf &hs, const TagBuf &cs,
                                   uint32_t tag) {
  constexpr int H4 = H / 4;
  const int total = r1 * H4;
  for (int e = blockIdx.x * kFwdThreads + threadIdx.x; e < total; e += gridDim.x * kFwdThreads) {
    const int r = e / H4, c4 = e % H4;
    int xr;
    if (xrow) {
      xr = xrow[r];
    } else {
      const int v = a.level_nodes[r];
      xr = (v >= 0 && v < a.N) ? a.x_index[v] : -1;
      if (xr < -1 || xr >= a.x_rows) {
        raise_status(a.status, CORTEX_ST_INPUT_RANGE);
        xr = -1;
      }
    }
    const float4 v = xr >= 0 ? *(const float4 *)&a.x_table[(size_t)xr * H + 4 * c4] : make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4 *)&a.h[(size_t)e * 4] = v;
    if (kWithC) *(float4 *)&a.c[(size_t)e * 4] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (a.ablate & 2) {
      hs.store1((uint32_t)e * 4u + 0u, v.x, tag);
      hs.store1((uint32_t)e * 4u + 1u, v.y, tag);
      hs.store1((uint32_t)e * 4u + 2u, v.z, tag);
      hs.store1((uint32_t)e * 4u + 3u, v.w, tag);
      if (kWithC) {
#pragma unroll
        for (int q = 0; q < 4; ++q) cs.store1((uint32_t)e * 4u + q, 0.f, tag);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fused launch (cortex_tree_infer): every workgroup linearizes the batch in
// LDS itself (small_linearize), workgroup 0 also writes the linearization
// out, and the structure cache of the slice kernel is built from the LDS
// results, so the first level needs no global memory beyond the inputs.
// Dynamic LDS (ints): the cache (4N + 1), the input row by node id (N), then
// the linearizer's own arrays.  Leaf-input cells only (TreeRNN, N-ary TreeLSTM).
// ---------------------------------------------------------------------------
constexpr int kFusedPer = 4;                       // nodes per thread: N <= 2048

// Trace builds: workgroup 0 stamps the in-kernel linearizer's phases into
// slots 4.. of its kernel-wide trace row (entry, children loaded, heights,
// level offsets, sort); nullptr otherwise.
__device__ __forceinline__ uint64_t *fused_lin_stamps(const FwdArgs &a) {
#ifdef CORTEX_TRACE
  if (blockIdx.x == 0) return a.trace + (size_t)(kTraceLevels - 1) * kTraceSlots + 4;
#endif
  (void)a;
  return nullptr;
}
constexpr int kFusedMaxNodes = kFwdThreads * kFusedPer;

static size_t fused_lds_ints(int32_t N, int32_t K) {
  return (size_t)4 * N + 1 + (size_t)N + small_lin_ints<kFwdThreads>(N, K);
}

template <int CELL>
__device__ bool fused_setup(const FwdArgs &a, int *cache, int &L, const int *&off, const int *&codes,
                            const int *&xrow) {
  using SC = SrcCfg<CELL>;
  constexpr int SEGS = SC::SEGS;
  static_assert((SC::kLeafX && SEGS == 2) || (SC::kDag && SEGS == 3), "leaf-input or DAG cells");
  const int N = a.N, K = a.K, tid = threadIdx.x;
  int *xnode = cache + 4 * N + 1;
  int *lin = xnode + N;
  // the input row of every node id (leaf-input cells), requested before the
  // linearizer's loads
  int xi[kFusedPer];
#pragma unroll
  for (int k = 0; k < kFusedPer; ++k) {
    const int v = tid + k * kFwdThreads;
    xi[k] = (SC::kLeafX && v < N) ? a.x_index[v] : -1;
  }
  SmallLin m;
  L = small_linearize<kFwdThreads, kFusedPer>(a.children, N, K, a.status, lin, m, fused_lin_stamps(a));
  if (L == 0) return false;
  if (blockIdx.x == 0)
    small_lin_emit<kFwdThreads>(m, N, K, L, a.o_num_levels, a.o_height, a.o_level_offsets, a.o_level_nodes,
                                a.o_node_row, a.o_child_rows);
  CORTEX_TRACE_KERNEL(9);
  int *o = cache, *cd = cache + (L + 1), *xr = cd + SEGS * N;
  for (int i = tid; i <= L; i += kFwdThreads) o[i] = i < L ? m.lcount[i] : N;
  if constexpr (SC::kLeafX) {
#pragma unroll
    for (int k = 0; k < kFusedPer; ++k) {
      const int v = tid + k * kFwdThreads;
      if (v < N) {
        int x = xi[k];
        if (x < -1 || x >= a.x_rows) {
          raise_status(a.status, CORTEX_ST_INPUT_RANGE);
          x = -1;
        }
        xnode[v] = x;
      }
    }
    __syncthreads();
    for (int r = tid; r < N; r += kFwdThreads) xr[r] = xnode[m.order[r]];
    __syncthreads();
  }
  const int off1 = L > 1 ? m.lcount[1] : N;
  // source codes: a child row, or (a leaf child of a leaf-input cell) -2 -
  // its input row; DAG-RNN: segment 0 is the node's own input row, -2 - id
  for (int r = tid; r < N; r += kFwdThreads) {
    const int v = m.order[r];
    if (SC::kDag) cd[r * SEGS] = -2 - v;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      int c = -1;
      if (s < K) {
        const int ch = m.ch[v * K + s];
        c = ch < 0 ? -1 : m.nrow[ch];
      }
      if (SC::kLeafX && !(a.ablate & 2) && c >= 0 && c < off1) c = xr[c] >= 0 ? -2 - xr[c] : -1;
      cd[r * SEGS + (SC::kDag ? s + 1 : s)] = c;
    }
  }
  __syncthreads();
  CORTEX_TRACE_KERNEL(10);
  off = o;
  codes = cd;
  xrow = SC::kLeafX ? xr : nullptr;
  return true;
}

// The Structure<true> cache (off, crow, xrow) built the same way from an
// in-LDS linearization, for the kernels that read child rows (TreeRNN at
// H = 64, child-sum TreeLSTM, TreeGRU cells).  Dynamic LDS (ints) from
// `cache`: off (N + 1), crow (N*K), xrow (N), the input row by node id (N),
// then the linearizer's arrays.
__host__ __device__ inline size_t fused_struct_ints(int N, int K) {
  return (size_t)N + 1 + (size_t)N * K + 2 * (size_t)N + small_lin_ints<kFwdThreads>(N, K);
}

__device__ bool fused_structure(const FwdArgs &a, int *cache, Structure<true> &st, int &L) {
  const int N = a.N, K = a.K, tid = threadIdx.x;
  int *o = cache, *crow = o + (N + 1), *xr = crow + N * K, *xnode = xr + N, *lin = xnode + N;
  int xi[kFusedPer];
#pragma unroll
  for (int k = 0; k < kFusedPer; ++k) {
    const int v = tid + k * kFwdThreads;
    xi[k] = v < N ? a.x_index[v] : -1;
  }
  SmallLin m;
  L = small_linearize<kFwdThreads, kFusedPer>(a.children, N, K, a.status, lin, m, fused_lin_stamps(a));
  if (L == 0) return false;
  if (blockIdx.x == 0)
    small_lin_emit<kFwdThreads>(m, N, K, L, a.o_num_levels, a.o_height, a.o_level_offsets, a.o_level_nodes,
                                a.o_node_row, a.o_child_rows);
  for (int i = tid; i <= L; i += kFwdThreads) o[i] = i < L ? m.lcount[i] : N;
#pragma unroll
  for (int k = 0; k < kFusedPer; ++k) {
    const int v = tid + k * kFwdThreads;
    if (v < N) {
      int x = xi[k];
      if (x < -1 || x >= a.x_rows) {
        raise_status(a.status, CORTEX_ST_INPUT_RANGE);
        x = -1;
      }
      xnode[v] = x;
    }
  }
  __syncthreads();
  for (int r = tid; r < N; r += kFwdThreads) {
    const int v = m.order[r];
    xr[r] = xnode[v];
    for (int s = 0; s < K; ++s) {
      const int c = m.ch[v * K + s];
      crow[r * K + s] = c < 0 ? -1 : m.nrow[c];
    }
  }
  __syncthreads();
  st.off = o;
  st.crow = crow;
  st.xrow = xr;
  st.node = nullptr;
  st.K = K;
  return true;
}

// Operand fragment: four consecutive k of one tile row, either staged (two
// (value, tag) pairs of pairs in lo and hi) or plain (four floats in lo: an
// input row, or zeros for an absent source).  Each lane issues only the loads
// its source needs.
struct Frag {
  u32x4 lo, hi;
  __device__ __forceinline__ bool ready(uint32_t tag) const {
    return lo.y == tag && lo.w == tag && hi.y == tag && hi.w == tag;
  }
  __device__ __forceinline__ float4 value(bool staged) const {
    return make_float4(as_float(lo.x), as_float(staged ? lo.z : lo.y), as_float(staged ? hi.x : lo.z),
                       as_float(staged ? hi.z : lo.w));
  }
};

// ---------------------------------------------------------------------------
// TreeRNN, N-ary TreeLSTM and DAG-RNN.
//   A row of a tile = [h(slot 0) | h(slot 1)]        (TreeRNN, N-ary TreeLSTM)
//                   = [x | h(slot 0) | h(slot 1)]    (DAG-RNN)
// Wave w owns the columns [w*KW, (w+1)*KW) of A (zero beyond KA); in block b
// lane group g (lanes 16g .. 16g+15) takes the columns w*KW + 16b + 4g ..+3,
// so the four lane groups of a row read one 128-byte span of staged pairs
// with each pair of load instructions.
// ---------------------------------------------------------------------------
template <int CELL, int H, int J, bool kCached, bool kWeightsFromMemory = false, bool kFused = false>
__global__ void __launch_bounds__(kFwdThreads) slice_forward_kernel(FwdArgs a) {
  using D = Dims<CELL, H, J>;
  constexpr int GJ = D::GJ, MPAD = D::MPAD, NT = D::NT, LDW = D::LDW, KW = D::KW, NB = D::NB, KA = D::KA;
  constexpr bool kLeafInputs = CELL == CORTEX_TREE_RNN || CELL == CORTEX_NARY_TREELSTM;
  constexpr bool kLstm = CELL == CORTEX_NARY_TREELSTM;
  constexpr int EPI = kTileM * J;          // (row, unit) pairs of a tile
  // Gate rows beyond the last full 16-row MFMA tile: when only four remain
  // (N-ary TreeLSTM, J = 4: the u gate), an MFMA tile would be three-quarters
  // padding, so they are contracted on the vector ALU, from the same operand
  // registers, while the matrix cores run the full tiles.
  constexpr bool kVecTail = GJ % 16 == 4 && NT >= 2;
  constexpr int NTM = kVecTail ? NT - 1 : NT;    // MFMA tiles of gate rows
  constexpr int SEGS = SrcCfg<CELL>::SEGS;
  // A block's 16 columns never straddle two operand segments (H is a
  // multiple of 16), so the segment of block b is the same for the whole
  // wave; a wave's range touches at most two segments (KW <= H).
  static_assert(KA == SEGS * H && KA <= kFwdWaves * KW && KW <= H && H % 16 == 0, "block layout");

  __shared__ __attribute__((aligned(16))) float W_s[MPAD * LDW];
  __shared__ __attribute__((aligned(16))) float C_s[kFwdWaves * kTileM * MPAD];
  __shared__ float Z_s[kLstm ? kTileM * GJ : 1];
  __shared__ float bias_s[MPAD];
  __shared__ ChunkSrc chunk;
  extern __shared__ int cache[];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  // node group q's slices are workgroups q, q + Q, q + 2Q, ..., which
  // round-robin dispatch puts on the XCDs congruent to q modulo gcd(Q, 8)
  // (two XCDs for Q = 4) instead of spreading a group over all eight
  const int slice = blockIdx.x / a.Q, group = blockIdx.x % a.Q, Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N;
  const uint32_t tag = launch_tag(a.sync);     // read with the status: one round trip
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const TagBuf cs(a.cs, kLstm ? (uint32_t)N * H * 8 : 0u);
  // plain operand rows: the input table (leaf children) or the DAG inputs
  const InBuf xin(CELL == CELL_DAG ? (const void *)a.x : (const void *)a.x_table,
                  CELL == CELL_DAG ? (a.x ? (uint32_t)N * H * 4 : 0u)
                                   : (kLeafInputs && a.x_table ? (uint32_t)a.x_rows * H * 4 : 0u));
  // this wave's columns: segment sgA from column o0 within it, crossing into
  // segment sgA + 1 at block cross_b (NB when it does not)
  const int kw = wave * KW;
  const int sgA = kw / H, o0 = kw % H;
  const int cross_b = (H - o0) / 16 < NB ? (H - o0) / 16 : NB;

  CORTEX_TRACE_KERNEL(0);
  // the status, the weight slice and the cached linearization are requested
  // together: one memory round trip for all of them
  const int status0 = load_status(a.status);
  int L;
  const int *off, *codes, *xrow;
  if constexpr (kFused) {
    // the weight loads share their round trip with the children and input
    // rows the linearizer requests
    static_assert(kCached && !kWeightsFromMemory, "fused launches cache the structure");
    WeightRegs<CELL, H, J> wr;
    issue_weight_slice<CELL, H, J>(a, hbase, wr);
    const bool ok = fused_setup<CELL>(a, cache, L, off, codes, xrow);
    commit_weight_slice<CELL, H, J>(wr, W_s, bias_s);
    if (!ok || status0 != 0) return;
    __syncthreads();                  // the weight slice is in LDS before any tile reads it
    CORTEX_TRACE_KERNEL(1);
  } else {
    SrcRegs pf;
    {
      WeightRegs<CELL, H, J> wr;
      issue_weight_slice<CELL, H, J>(a, hbase, wr);
      prefetch_sources<CELL, kCached>(a, pf);
      commit_weight_slice<CELL, H, J>(wr, W_s, bias_s);
    }
    if (status0 != 0) return;
    CORTEX_TRACE_KERNEL(1);
    if (!setup_sources<CELL, kCached>(a, pf, cache, L, off, codes, xrow)) return;
  }
  CORTEX_TRACE_KERNEL(2);
  if (!mark_entered(a.sync, tag, a.status)) return;
  const int off1 = off[1];
  int gave_up = 0;

  for (int l = a.level_lo; l < L && l < a.level_hi; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = off[l], r1 = off[l + 1];
    if (!kCached && (r1 < r0 || r1 > N || (l == 0 && r0 != 0))) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    if (kLeafInputs && l == 0) {
      write_leaf_outputs<H, kLstm>(a, kCached ? xrow : nullptr, r1, hs, cs, tag);
      continue;
    }
    const int ntile = (r1 - r0 + kTileM - 1) / kTileM;
    int u0 = ((group - l) % Q + Q) % Q;            // first tile of the current chunk

    // source code of tile u, row i, segment sg (cached, or the staged chunk)
    auto code_of = [&](int u, int i, int sg) __attribute__((always_inline)) -> int {
      if (kCached) return codes[(r0 + u * kTileM + i) * SEGS + sg];
      return chunk.code[(u - u0) / Q][i][sg];
    };
    auto code_b = [&](const int (&cd)[2], int b) __attribute__((always_inline)) -> int {
      return b >= cross_b ? cd[1] : cd[0];
    };
    auto col_b = [&](int b) __attribute__((always_inline)) -> int {   // this lane's first column in block b
      return (b >= cross_b ? o0 + 16 * b - H : o0 + 16 * b) + 4 * g4;
    };

    // Operands of tile u for this lane: fragments f, the row's source codes
    // cd (this lane's segment and the next), and (N-ary) the staged memory
    // cells cc of pair tid's non-leaf children (elements ce).
    auto issue = [&](int u, Frag (&f)[NB], int (&cd)[2], u32x2 (&cc)[2], int (&ce)[2]) __attribute__((always_inline)) {
      const int row = r0 + u * kTileM + i16;
      cd[0] = cd[1] = -1;
      if (row < r1 && sgA < SEGS) {
        cd[0] = code_of(u, i16, sgA);
        if (cross_b < NB && sgA + 1 < SEGS) cd[1] = code_of(u, i16, sgA + 1);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int c = code_b(cd, b), o = col_b(b);
        if (c >= 0) {
          const uint32_t so = (uint32_t)(c * H + o) * 8u;
          f[b].lo = hs.load2_at(so);
          f[b].hi = hs.load2_at(so + 16u);
        } else {
          // both halves written on both paths: a store to a selected half
          // would force the fragments out of registers
          f[b].lo = xin.load4(c <= -2 ? (uint32_t)(((-2 - c) * H + o) * 4) : kNoSource);
          f[b].hi = u32x4{0u, 0u, 0u, 0u};
        }
      }
      if (kLstm) {
        const int prow = r0 + u * kTileM + tid / J;
        const bool live = tid < EPI && prow < r1;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int c = live ? code_of(u, tid / J, s) : -1;
          ce[s] = c >= 0 ? c * H + hbase + tid % J : -1;
          cc[s] = cs.load1_at(ce[s] >= 0 ? (uint32_t)ce[s] * 8u : kNoSource);
        }
      }
    };
    auto all_ready = [&](const Frag (&f)[NB], const int (&cd)[2], const u32x2 (&cc)[2],
                         const int (&ce)[2]) __attribute__((always_inline)) -> bool {
      bool r = true;
#pragma unroll
      for (int b = 0; b < NB; ++b) r = r && (code_b(cd, b) < 0 || f[b].ready(tag));
      if (kLstm) {
#pragma unroll
        for (int s = 0; s < 2; ++s) r = r && (ce[s] < 0 || cc[s].y == tag);
      }
      return r;
    };

    // One tile: wait for its staged operands, request the next tile's, contract,
    // apply the gates, write the states.
    auto process = [&](int u, Frag (&f)[NB], int (&cd)[2], u32x2 (&cc)[2], int (&ce)[2], bool more,
                       Frag (&fn)[NB], int (&cdn)[2], u32x2 (&ccn)[2], int (&cen)[2]) __attribute__((always_inline)) {
      CORTEX_TRACE_POINT(l, 1);
      if (!gave_up && !all_ready(f, cd, cc, ce)) {
        const uint64_t t0 = wall_clock64();
        for (;;) {
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            const int c = code_b(cd, b);
            if (c >= 0 && !f[b].ready(tag)) {
              const uint32_t so = (uint32_t)(c * H + col_b(b)) * 8u;
              f[b].lo = hs.load2_at(so);
              f[b].hi = hs.load2_at(so + 16u);
            }
          }
          if (kLstm) {
#pragma unroll
            for (int s = 0; s < 2; ++s)
              if (ce[s] >= 0 && cc[s].y != tag) cc[s] = cs.load1_at((uint32_t)ce[s] * 8u);
          }
          const int stv = load_status(a.status);
          if (all_ready(f, cd, cc, ce)) break;
          if (stv != 0) {
            gave_up = 1;
            break;
          }
          if (wall_clock64() - t0 > a.timeout) {
            raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
            gave_up = 1;
            break;
          }
        }
      }
      CORTEX_TRACE_POINT(l, 2);
      if (more) issue(u + Q, fn, cdn, ccn, cen);   // in flight during this tile's contraction
      // ---- contraction: partial sums of this wave's k range ----
      floatx4 acc0[NT], acc1[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc0[nt] = acc1[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
      // vector-ALU rows: this lane's row i16 over its 4 NB columns, for the
      // four gate rows 16 NTM .. +3
      float tail[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!kWeightsFromMemory) {
        const float *brow = &W_s[i16 * LDW + kw + 4 * g4];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const float4 av = f[b].value(code_b(cd, b) >= 0);
#pragma unroll
          for (int nt = 0; nt < NTM; ++nt) {
            const float4 bv = *(const float4 *)(brow + nt * 16 * LDW + 16 * b);
            if (b & 1) acc1[nt] = mfma_k16(av, bv, acc1[nt]);
            else acc0[nt] = mfma_k16(av, bv, acc0[nt]);
          }
          if constexpr (kVecTail) {
            const float *trow = &W_s[16 * NTM * LDW + kw + 16 * b + 4 * g4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float4 w = *(const float4 *)(trow + q * LDW);
              tail[q] = fmaf(av.x, w.x, fmaf(av.y, w.y, fmaf(av.z, w.z, fmaf(av.w, w.w, tail[q]))));
            }
          }
        }
      } else {
        // ablation: no model persistence; the same weight-slice values,
        // read from the weight tensors at every tile
        float4 bw[NB][NTM];
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int nt = 0; nt < NTM; ++nt) bw[b][nt] = weight_slice_at<CELL, H, J>(a, hbase, nt * 16 + i16, kw + 16 * b + 4 * g4);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const float4 av = f[b].value(code_b(cd, b) >= 0);
#pragma unroll
          for (int nt = 0; nt < NTM; ++nt) {
            if (b & 1) acc1[nt] = mfma_k16(av, bw[b][nt], acc1[nt]);
            else acc0[nt] = mfma_k16(av, bw[b][nt], acc0[nt]);
          }
          if constexpr (kVecTail) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float4 w = weight_slice_at<CELL, H, J>(a, hbase, 16 * NTM + q, kw + 16 * b + 4 * g4);
              tail[q] = fmaf(av.x, w.x, fmaf(av.y, w.y, fmaf(av.z, w.z, fmaf(av.w, w.w, tail[q]))));
            }
          }
        }
      }
      CORTEX_TRACE_WAVE(l);
      // The next tile's loads stay in flight through this tile's epilogue
      // (vector memory operations retire in order, so their first use
      // waits for them alone).
#pragma unroll
      for (int nt = 0; nt < NTM; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          C_s[(wave * kTileM + 4 * g4 + v) * MPAD + nt * 16 + i16] = acc0[nt][v] + acc1[nt][v];
      if constexpr (kVecTail) {
        // the four lanes of row i16 (lane groups g4) hold disjoint column sets
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          tail[q] += __shfl_xor(tail[q], 16);
          tail[q] += __shfl_xor(tail[q], 32);
        }
        if (g4 == 0)
          *(float4 *)&C_s[(wave * kTileM + i16) * MPAD + 16 * NTM] = make_float4(tail[0], tail[1], tail[2], tail[3]);
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 3);
      // ---- gates: one thread per (row, gate row) sums the wave partials
      //      and applies the nonlinearity; TreeRNN / DAG-RNN rows are done
      //      here, N-ary TreeLSTM combines the gates below ----
      for (int p = tid; p < kTileM * GJ; p += kFwdThreads) {
        const int i = p / GJ, m = p % GJ;
        float sum = bias_s[m];
#pragma unroll
        for (int w = 0; w < kFwdWaves; ++w) sum += C_s[(w * kTileM + i) * MPAD + m];
        if constexpr (kLstm) {
          Z_s[p] = m >= 4 * J ? tanh_f(sum) : sigmoidf(sum);      // gates (i, f_l, f_r, o | u)
        } else {
          const int row = r0 + u * kTileM + i;
          if (row < r1) {
            const uint32_t el = (uint32_t)(row * H + hbase + m);
            const float hv = tanh_f(sum);
            hs.store1(el, hv, tag);
            a.h[el] = hv;
          }
        }
      }
      if constexpr (kLstm) {
        __syncthreads();
        const int row = r0 + u * kTileM + tid / J;
        if (tid < EPI && row < r1) {
          const int j = tid % J;
          const float *z = &Z_s[(tid / J) * GJ];
          const float cn = z[j] * z[4 * J + j] + z[J + j] * as_float(cc[0].x) + z[2 * J + j] * as_float(cc[1].x);
          const float hv = z[3 * J + j] * tanh_f(cn);
          const uint32_t el = (uint32_t)(row * H + hbase + j);
          cs.store1(el, cn, tag);
          hs.store1(el, hv, tag);
          a.c[el] = cn;
          a.h[el] = hv;
        }
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 4);
    };

    // Two operand sets in turn: the next tile's loads are in flight while
    // the current tile is computed, with no register copies between tiles.
    Frag fa[NB], fb[NB];
    int cda[2], cdb[2], cea[2] = {-1, -1}, ceb[2] = {-1, -1};
    u32x2 cca[2], ccb[2];
    for (; u0 < ntile; u0 += Q * kChunkTiles) {
      const int u_last = min(ntile - 1, u0 + Q * (kChunkTiles - 1));
      if (!kCached) {
        __syncthreads();                // the previous chunk's codes are no longer read
        stage_chunk_codes<CELL>(a, chunk, u0, (u_last - u0) / Q + 1, Q, r0, r1, off1);
        __syncthreads();
      }
      issue(u0, fa, cda, cca, cea);
      CORTEX_TRACE_POINT(l, 6);
      for (int u = u0;;) {
        bool more = u + Q <= u_last;
        process(u, fa, cda, cca, cea, more, fb, cdb, ccb, ceb);
        u += Q;
        if (!more) break;
        more = u + Q <= u_last;
        process(u, fb, cdb, ccb, ceb, more, fa, cda, cca, cea);
        u += Q;
        if (!more) break;
      }
    }
    CORTEX_TRACE_POINT(l, 5);
    if (__syncthreads_or(gave_up)) return;
    if (a.level_barrier && !grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout)) return;
  }
  CORTEX_TRACE_KERNEL(3);
  if (a.retire) retire_tag(a.sync, tag, a.status, a.timeout);
}

// ---------------------------------------------------------------------------
// TreeRNN at H = 64 in one workgroup with every state in LDS.
//   h = tanh(W [h(slot 0); h(slot 1)] + b),  leaf h = its input row.
// The whole cell fits one CU: wave w holds W[16 (w & 3) .., (w >> 2) * 64 ..]
// (its 16 output units x the 64 columns of child slot w >> 2) in registers,
// and the h row of every node stays in LDS, so a level reads its children
// from LDS and one barrier orders consecutive levels; nothing goes through
// global memory between levels, and the states are written out once at the
// end.  Used while the rows fit the LDS budget.
// ---------------------------------------------------------------------------
constexpr int kLdsH = 64;
constexpr int kLdsHStride = kLdsH + 4;        // h row stride in LDS
constexpr int kLdsMaxRows = 320;              // rows kept in LDS

template <bool kFused = false>
__global__ void __launch_bounds__(kFwdThreads) tree_rnn_lds_kernel(FwdArgs a) {
  constexpr int H = kLdsH, LDH = kLdsHStride, NB = H / 16;
  constexpr int EPI = kTileM * H / kFwdThreads;
  __shared__ __attribute__((aligned(16))) float C_s[2][kTileM][H + 4];
  __shared__ float bias_s[H];
  extern __shared__ __attribute__((aligned(16))) float dyn_s[];   // h rows, then the structure cache

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int nt = wave & 3, kh = wave >> 2;     // this wave's output units and child slot
  const int N = a.N;
  float *h_s = dyn_s;
  int *cache = (int *)(dyn_s + (size_t)N * LDH);

  CORTEX_TRACE_KERNEL(0);
  const int status0 = load_status(a.status);  // one round trip with the weight loads
  // wr[b] = W[16 nt + i16][64 kh + 16 b + 4 g4 .. +3]
  float4 wr[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    wr[b] = *(const float4 *)(a.W + (size_t)(16 * nt + i16) * 2 * H + kh * H + 16 * b + 4 * g4);
  if (tid < H) bias_s[tid] = a.b[tid];
  Structure<true> st;
  int L;
  if constexpr (kFused) {
    // the batch is linearized here (its loads share the weights' round trip)
    if (!fused_structure(a, cache, st, L) || status0 != 0) return;
    CORTEX_TRACE_KERNEL(1);
  } else {
    if (status0 != 0) return;
    CORTEX_TRACE_KERNEL(1);
    if (!setup_structure<true, true, false>(a, cache, st, L)) return;
  }
  CORTEX_TRACE_KERNEL(2);

  // level 0: the leaves are their input rows (zeros without one)
  const int off1 = st.offset(1 < L ? 1 : L);
  CORTEX_TRACE_POINT(0, 0);
  for (int e = tid; e < off1 * (H / 4); e += kFwdThreads) {
    const int r = e / (H / 4), c4 = e % (H / 4);
    const int xr = st.input_row(r);
    const float4 v = xr >= 0 ? *(const float4 *)&a.x_table[(size_t)xr * H + 4 * c4] : make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4 *)&h_s[r * LDH + 4 * c4] = v;
  }
  __syncthreads();
  CORTEX_TRACE_POINT(0, 5);

  for (int l = 1; l < L; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = st.offset(l), r1 = st.offset(l + 1);
    for (int rowbase = r0; rowbase < r1; rowbase += kTileM) {
      const int row = rowbase + i16;
      const int cr = row < r1 ? st.child(row, kh) : -1;
      float4 av[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        av[b] = cr >= 0 ? *(const float4 *)&h_s[cr * LDH + 16 * b + 4 * g4] : make_float4(0.f, 0.f, 0.f, 0.f);
      CORTEX_TRACE_POINT(l, 2);
      floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (b & 1) acc1 = mfma_k16(av[b], wr[b], acc1);
        else acc0 = mfma_k16(av[b], wr[b], acc0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) C_s[kh][4 * g4 + v][16 * nt + i16] = acc0[v] + acc1[v];
      __syncthreads();
      CORTEX_TRACE_POINT(l, 3);
#pragma unroll
      for (int e = 0; e < EPI; ++e) {
        const int p = tid + e * kFwdThreads, i = p / H, j = p % H;
        const int r = rowbase + i;
        if (r < r1) h_s[r * LDH + j] = tanh_f(bias_s[j] + C_s[0][i][j] + C_s[1][i][j]);
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 4);
    }
    CORTEX_TRACE_POINT(l, 5);
  }
  // every state leaves LDS once, coalesced (no global store inside the
  // level loop, whose barriers would otherwise wait for them)
  for (int e = tid; e < N * (H / 4); e += kFwdThreads) {
    const int r = e / (H / 4), c4 = e % (H / 4);
    *(float4 *)&a.h[(size_t)r * H + 4 * c4] = *(const float4 *)&h_s[r * LDH + 4 * c4];
  }
  CORTEX_TRACE_KERNEL(3);
}

// ---------------------------------------------------------------------------
// DAG-RNN at H = 256 with four hidden slices of 64 units:
//   h(v) = tanh(W x(v) + U_0 h(slot 0) + U_1 h(slot 1) + b).
// Fewer, wider slices than the kernel above: every slice re-reads the child
// rows it contracts, so four slices move a quarter of the operand bytes of
// sixteen.  Each wave keeps its 64 recurrent columns x 64 units of U_0 / U_1
// in registers for the whole launch and the input weights W sit in LDS.  When
// the grid is a multiple of 32, the four slices of node group q are
// workgroups 32m + r + 8s (r = q mod 8, m = q div 8, s = 0..3), which
// round-robin dispatch places on one XCD, so the input row of a node is
// fetched into one L2 once.
//
// Work is done in steps: a step is up to two of the group's 16-row tiles of
// one level (group q owns the tiles u of level l with u = q - l mod Q, so a
// level of up to 2Q tiles is one step per group).  The tiles of a step share
// one wait, one cross-wave reduction and one epilogue, and every weight
// fragment is read once for both tiles.  Per step, wave w
//   1. contracts input columns [32w, 32w+32) (requested one step earlier;
//      they depend on no child); between the MFMA steps of the first half it
//      requests the next step's input fragments, and between those of the
//      second half the child-state fragments of its recurrent columns
//      [64w, 64w+64) of [h(slot 0) | h(slot 1)] for every row of the step,
//   2. waits until every fragment it read carries this launch's tag,
//   3. contracts the recurrent columns;
// the eight partial sums then meet in LDS and the workgroup applies tanh and
// writes the step's rows.  The next step's input fragments are complete
// before the stores are issued, so no wait of the next step covers them.
// A level of at most Q/2 tiles is split finer: each of its tiles is a half
// step of two groups, one per half of the slice's units, so the narrow first
// and last levels of a batch, whose chain of waits sets the pace, take half
// the contraction time per group.  At entry each workgroup lists its steps of
// every level with their operand sources in LDS, so the level loop never
// goes back to the linearization in memory; a group with more steps than the
// list holds (60) lists them a chunk at a time, the next chunk once it has
// run the previous one.
// ---------------------------------------------------------------------------
constexpr int kDagH = 256, kDagJ = 64, kDagS = kDagH / kDagJ;
constexpr int kDagWideMinRows = 6144;              // default choice of this kernel (measured crossover)
constexpr int kDagStepTiles = 2;                   // tiles per step
constexpr int kDagStepRows = kDagStepTiles * kTileM;
// level, level start, first row of tile 0, first row of tile 1 (-1: none),
// level end, units (0: the slice's 64, 1: its first 32, 2: its last 32),
// then codes[32][3]: -2 - node id (input row) or -1, child rows
constexpr int kDagStepHead = 6;
constexpr int kDagStepInts = kDagStepHead + kDagStepRows * 3;
constexpr int kDagStepCap = 60;                    // steps per workgroup list (dynamic LDS)
constexpr size_t kDagListBytes = (size_t)kDagStepCap * kDagStepInts * sizeof(int);

// Exclusive prefix sum of one value per thread over the workgroup; wsum
// holds kFwdWaves + 1 ints of LDS.  Returns the exclusive sum, *total the sum.
__device__ __forceinline__ int block_excl_scan(int v, int *wsum, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < kFwdWaves; ++w) {
      const int t = wsum[w];
      wsum[w] = run;
      run += t;
    }
    wsum[kFwdWaves] = run;
  }
  __syncthreads();
  const int ex = wsum[wave] + x - v;
  *total = wsum[kFwdWaves];
  __syncthreads();
  return ex;
}

// Tiles of group `group` at a level of ntile tiles; returns their count.
// Normally the tiles u = uf, uf + Q, ... with uf = (group - l) mod Q, whole
// (half = 0).  A level of at most Q/2 tiles (Q even) gives each tile to two
// groups, each computing half of its slice's units, so the tile's
// contraction is split over twice the compute units: group q takes tile
// (q - l) mod Q as half 1 (the first 32 units) or tile (q - l + Q/2) mod Q
// as half 2 (the last 32); at most one of the two exists.
__device__ __forceinline__ int dag_group_tiles(int group, int l, int Q, int ntile, int &uf, int &half) {
  const int u1 = ((group - l) % Q + Q) % Q;
  half = 0;
  uf = u1;
  if (Q % 2 == 0 && 2 * ntile <= Q) {
    const int u2 = (u1 + Q / 2) % Q;
    if (u1 < ntile) {
      half = 1;
      return 1;
    }
    if (u2 < ntile) {
      uf = u2;
      half = 2;
      return 1;
    }
    return 0;
  }
  return u1 < ntile ? (ntile - 1 - u1) / Q + 1 : 0;
}

// The row of slot (t, i) of a step record, or -1 when the slot is empty.
__device__ __forceinline__ int dag_slot_row(const int *st, int slot) {
  const int base = st[2 + slot / kTileM], row = base + slot % kTileM;
  return (base >= 0 && row < st[4]) ? row : -1;
}

// Stores the operand sources of a slot from its row's node id v and child
// rows c0, c1 (read when live, i.e. the slot holds a row), validated as the
// forward requires (a child lies below its row's level); returns false when
// the linearization is inconsistent.
__device__ __forceinline__ bool dag_store_codes(const FwdArgs &a, int *st, int slot, bool live, int v, int c0, int c1) {
  const int lstart = st[1];
  int *cd = &st[kDagStepHead + slot * 3];
  if (!live) v = c0 = c1 = -1;
  bool ok = !live || (v >= 0 && v < a.N);
  cd[0] = (v >= 0 && v < a.N) ? -2 - v : -1;
  if (c0 < -1 || c0 >= lstart) {
    ok = false;
    c0 = -1;
  }
  if (c1 < -1 || c1 >= lstart) {
    ok = false;
    c1 = -1;
  }
  cd[1] = c0;
  cd[2] = c1;
  return ok;
}

// Hoisted input products of the DAG-RNN at H = 256 (the ablation of the
// fused input part; Sec. 7.1 computes them with one matrix product before the
// recursion): pre[r][u] = sum_k x[node(r)][k] W[u][k] + b[u] for every row r,
// in row order.  Workgroup (row block m, slice s) computes rows
// [128m, 128m + 128) x units [64s, 64s + 64): each wave 16 rows, its input
// fragments in registers, the slice of W in LDS, fp32 MFMA.  With a grid that
// is a multiple of 32, the four slices of a row block are workgroups
// 32m' + r + 8s (m = 8m' + r), which round-robin dispatch places on one XCD.
__global__ void __launch_bounds__(kFwdThreads) dag_input_gemm_kernel(FwdArgs a) {
  constexpr int H = kDagH, J = kDagJ, NT = J / 16, NB = H / 16, LDX = H + 4;
  __shared__ __attribute__((aligned(16))) float W_s[J * LDX];
  __shared__ float bias_s[J];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int bid = blockIdx.x;
  const bool xcd_map = (gridDim.x & 31) == 0;
  const int slice = xcd_map ? ((bid >> 3) & 3) : bid % kDagS;
  const int block = xcd_map ? ((bid & 7) + 8 * (bid >> 5)) : bid / kDagS;
  const int N = a.N, hbase = slice * J;
  const int r0 = block * (kFwdWaves * kTileM);
  if (r0 >= N || load_status(a.status) != 0) return;
  // input fragments of row r0 + 16 wave + i16: x[node][16 b + 4 g4 .. +3]
  const int r = r0 + kTileM * wave + i16;
  const int v = r < N ? a.level_nodes[r] : -1;
  const InBuf xin(a.x, (uint32_t)N * H * 4);
  const uint32_t xo = (v >= 0 && v < N) ? (uint32_t)(v * H + 4 * g4) * 4u : kNoSource;
  u32x4 xf[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) xf[b] = xin.load4(xo + 64u * b);
  {
    constexpr int PER = J * H / 4 / kFwdThreads;
    float4 w[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads;
      w[k] = *(const float4 *)(a.W + (size_t)(hbase + idx / (H / 4)) * H + 4 * (idx % (H / 4)));
    }
    if (tid < J) bias_s[tid] = a.b[hbase + tid];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads;
      *(float4 *)&W_s[(idx / (H / 4)) * LDX + 4 * (idx % (H / 4))] = w[k];
    }
  }
  __syncthreads();
  floatx4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float *bx = &W_s[i16 * LDX + 4 * g4];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float4 wv[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wv[nt] = *(const float4 *)(bx + nt * 16 * LDX + 16 * b);
    mfma_k16_xn<NT>(as_float4(xf[b]), wv, acc);
  }
  // lane (i16, g4) holds rows 4 g4 .. 4 g4 + 3 of the wave's 16, column 16 nt + i16
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = r0 + kTileM * wave + 4 * g4 + e;
      if (row < N) a.pre[(size_t)row * H + hbase + 16 * nt + i16] = acc[nt][e] + bias_s[16 * nt + i16];
    }
}

template <bool kHoisted>
__global__ void __launch_bounds__(kFwdThreads) dag_slice64_kernel(FwdArgs a) {
  constexpr int H = kDagH, J = kDagJ, NT = J / 16;
  constexpr int KX = H / kFwdWaves, NBX = KX / 16;          // input columns per wave, 16-blocks
  constexpr int KR = 2 * H / kFwdWaves, NBR = KR / 16;      // recurrent columns per wave, 16-blocks
  constexpr int LDX = H + 4;                                // W row stride in LDS
  // partial sums: C_s[wave][tile][column][16 rows], the four 16-byte row
  // quarters of column c stored in the order q ^ ((c >> 2) & 3), so the
  // 16-byte accesses of 16 consecutive columns meet 64 distinct banks
  constexpr int MT = kDagStepTiles;
  constexpr int SI = kDagStepInts;
  constexpr int EPI = MT * kTileM * J / kFwdThreads;        // outputs per thread per full step
  static_assert(NBX * 16 == KX && NBR * 16 == KR && EPI * kFwdThreads == MT * kTileM * J, "tiling");
  static_assert(KR == 64 && H % KR == 0, "a wave's recurrent columns lie in one child slot");

  __shared__ __attribute__((aligned(16))) float Wx_s[kHoisted ? 4 : J * LDX];
  __shared__ __attribute__((aligned(16))) float C_s[kFwdWaves * MT * J * kTileM];
  __shared__ int stop_s;
  __shared__ float bias_s[J];
  __shared__ int wsum[kFwdWaves + 1];
  extern __shared__ int list[];               // [kDagStepCap][kDagStepInts]

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int bid = blockIdx.x;
  const bool xcd_map = (gridDim.x & 31) == 0;
  const int slice = xcd_map ? ((bid >> 3) & 3) : bid % kDagS;
  const int group = xcd_map ? ((bid & 7) + 8 * (bid >> 5)) : bid / kDagS;
  const int Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N;
  const uint32_t tag = launch_tag(a.sync);     // read with the status: one round trip
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const InBuf xin(a.x, kHoisted ? 0u : (uint32_t)N * H * 4);
  const InBuf pin(a.pre, kHoisted ? (uint32_t)N * H * 4 : 0u);
  const int rslot = wave >> 2;                 // child slot of this wave's recurrent columns
  const int rcol = KR * (wave & 3);            // their first column within that child's h
  const int xcol = KX * wave;                  // this wave's first input column

  CORTEX_TRACE_KERNEL(0);
  // The structure is read first and the weights (192 KB per workgroup, the
  // longest transfer of the entry) are requested once the step list is
  // known, after the operand sources' loads: vector loads complete in order,
  // so weights requested first would hold back every structure read behind
  // them.
  const int status0 = load_status(a.status);
  const int L = *a.num_levels;
  if (tid == 0) stop_s = 0;
  if (status0 != 0) return;
  if (L < 1 || L > N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }

  // ---- this group's steps of every level, one level per thread per round:
  // the list holds steps [first, first + kDagStepCap) of them; returns the
  // group's step count.  A group with more steps runs them in chunks,
  // listing the next chunk once it has run the previous one.
  auto list_steps = [&](int first, int &bad) __attribute__((always_inline)) -> int {
    int total = 0;
    for (int lb = 0; lb < L; lb += kFwdThreads) {
      const int l = lb + tid;
      int nst = 0, r0 = 0, r1 = 0, uf = 0, cnt = 0, half = 0;
      if (l < L) {
        r0 = a.level_offsets[l];
        r1 = a.level_offsets[l + 1];
        const bool ok = r0 >= 0 && r1 >= r0 && r1 <= N && (l != 0 || r0 == 0) && (l != L - 1 || r1 == N);
        if (!ok) bad = 1;
        const int ntile = (ok && l >= a.level_lo && l < a.level_hi) ? (r1 - r0 + kTileM - 1) / kTileM : 0;
        cnt = dag_group_tiles(group, l, Q, ntile, uf, half);
        nst = (cnt + MT - 1) / MT;
      }
      int round_total;
      const int pos = total + block_excl_scan(nst, wsum, &round_total) - first;
      for (int j = max(0, -pos); j < nst && pos + j < kDagStepCap; ++j) {
        int *st = &list[(pos + j) * SI];
        st[0] = l;
        st[1] = r0;
        st[2] = r0 + kTileM * (uf + (MT * j) * Q);
        st[3] = MT * j + 1 < cnt ? r0 + kTileM * (uf + (MT * j + 1) * Q) : -1;
        st[4] = r1;
        st[5] = half;
      }
      total += round_total;
    }
    return total;
  };
  int bad = 0;
  const int total = list_steps(0, bad);
  // (each level's end is the next level's start, so the levels tile [0, N))
  if (__syncthreads_or(bad)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  int listed = min(total, kDagStepCap);        // steps in the list
  // operand sources of every listed slot: requested now, stored below
  constexpr int kFillPer = (kDagStepCap * kDagStepRows + kFwdThreads - 1) / kFwdThreads;
  int frow[kFillPer], fv[kFillPer], f0[kFillPer], f1[kFillPer];
#pragma unroll
  for (int k = 0; k < kFillPer; ++k) {
    const int idx = tid + k * kFwdThreads;
    frow[k] = idx < listed * kDagStepRows ? dag_slot_row(&list[(idx / kDagStepRows) * SI], idx % kDagStepRows) : -1;
    fv[k] = f0[k] = f1[k] = -1;
    if (frow[k] >= 0) {
      fv[k] = a.level_nodes[frow[k]];
      f0[k] = a.child_rows[(size_t)frow[k] * 2];
      f1[k] = a.child_rows[(size_t)frow[k] * 2 + 1];
    }
  }
  // recurrent weights: wr[b][nt] = U_rslot[hbase + 16 nt + i16][rcol + 16 b + 4 g4 .. +3]
  float4 wr[NBR][NT];
#pragma unroll
  for (int b = 0; b < NBR; ++b)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      wr[b][nt] = *(const float4 *)(a.U + ((size_t)rslot * H + hbase + 16 * nt + i16) * H + rcol + 16 * b + 4 * g4);
  constexpr int ITEMS = J * H / 4, PER = kHoisted ? 1 : ITEMS / kFwdThreads;
  float4 v[PER];
  if constexpr (!kHoisted) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads;
      v[k] = *(const float4 *)(a.W + (size_t)(hbase + idx / (H / 4)) * H + 4 * (idx % (H / 4)));
    }
    if (tid < J) bias_s[tid] = a.b[hbase + tid];
  }
#pragma unroll
  for (int k = 0; k < kFillPer; ++k) {
    const int idx = tid + k * kFwdThreads;
    if (idx < listed * kDagStepRows &&
        !dag_store_codes(a, &list[(idx / kDagStepRows) * SI], idx % kDagStepRows, frow[k] >= 0, fv[k], f0[k], f1[k]))
      bad = 1;
  }
  if constexpr (!kHoisted) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads;
      *(float4 *)&Wx_s[(idx / (H / 4)) * LDX + 4 * (idx % (H / 4))] = v[k];
    }
  }
  if (__syncthreads_or(bad)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  CORTEX_TRACE_KERNEL(1);
  CORTEX_TRACE_KERNEL(2);
  if (!mark_entered(a.sync, tag, a.status)) return;
  int gave_up = 0;

  // input fragments of a step's rows (tile t, row i16): x[node][xcol + 16 b + 4 g4 .. +3]
  // (live false: every load reads zeros, so a step without a successor still
  // issues the same loads and the waits after them keep fixed counts)
  auto x_offsets = [&](const int *st, bool live, uint32_t (&xo)[MT]) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int base = st[2 + t];
      const int xc = (live && base >= 0 && base + i16 < st[4]) ? st[kDagStepHead + (t * kTileM + i16) * 3] : -1;
      xo[t] = xc <= -2 ? (uint32_t)(((-2 - xc) * H + xcol + 4 * g4) * 4) : kNoSource;
    }
  };
  auto issue_x = [&](const int *st, u32x4 (&xv)[MT][NBX], bool live) __attribute__((always_inline)) {
    uint32_t xo[MT];
    x_offsets(st, live, xo);
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int b = 0; b < NBX; ++b) xv[t][b] = xin.load4(xo[t] + 64u * b);
  };

  // One step.  half_c: the step's units as a compile-time constant (0: the
  // slice's 64, 1: its first 32, 2: its last 32; a half step has one tile);
  // xc: its input fragments (requested earlier); nst: the next step
  // (nullptr: none), whose input fragments go to xn.  Returns true when the
  // kernel must stop.
  auto run_step = [&](auto half_c, const int *st, const u32x4 (&xc)[MT][NBX], const int *nst,
                      u32x4 (&xn)[MT][NBX]) __attribute__((always_inline)) -> bool {
    constexpr int kHalf = decltype(half_c)::value;
    constexpr int NT0 = kHalf == 2 ? NT / 2 : 0;         // first n-tile of the step's units
    constexpr int NTS = kHalf == 0 ? NT : NT / 2;        // n-tiles of the step's units
    const int l = st[0], lend = st[4];
    const bool two = kHalf == 0 && st[3] >= 0;
    // epilogue thread: unit ej (within the slice) of row quarter eq of tile
    // et; a whole step uses every thread, a half step the first 128
    const int ej = kHalf == 0 ? (tid & (J - 1)) : J / 2 * (kHalf - 1) + (tid & (J / 2 - 1));
    const int et = kHalf == 0 ? tid / (J * 4) : 0;
    const int eq = kHalf == 0 ? (tid / J) & 3 : (tid / (J / 2)) & 3;
    const bool elive = kHalf == 0 ? (et == 0 || two) : tid < J / 2 * 4;
    Frag hv[MT][NBR];
    int cr[MT];
    uint32_t ho[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int base = st[2 + t];
      cr[t] = (base >= 0 && base + i16 < lend) ? st[kDagStepHead + (t * kTileM + i16) * 3 + 1 + rslot] : -1;
      ho[t] = cr[t] >= 0 ? (uint32_t)(cr[t] * H + rcol + 4 * g4) * 8u : kNoSource;
    }
    floatx4 acc[MT][NT];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[t][nt] = floatx4{0.f, 0.f, 0.f, 0.f};
    // the accumulators and recurrent weights of the step's units
    auto step_acc = [&](int t) __attribute__((always_inline)) -> floatx4 (&)[NTS] {
      return *reinterpret_cast<floatx4 (*)[NTS]>(&acc[t][NT0]);
    };
    auto step_wr = [&](int b) __attribute__((always_inline)) -> const float4 (&)[NTS] {
      return *reinterpret_cast<const float4 (*)[NTS]>(&wr[b][NT0]);
    };
    float pv[4];                             // hoisted: W x + b of the thread's four outputs
    if constexpr (kHoisted) {
      // 1. (hoisted) the step's input products, computed before the level
      // loop, for the epilogue's four outputs of this thread, then every
      // child-state fragment of the step at once: there is no input part to
      // place them in
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = st[2 + et] + 4 * eq + v;
        pv[v] = as_float(pin.load1((elive && row < lend) ? (uint32_t)(row * H + hbase + ej) * 4u : kNoSource));
      }
#pragma unroll
      for (int k = 0; k < NBR; ++k) {
        hv[0][k].lo = hs.load2_at(ho[0] + 128u * k);
        hv[0][k].hi = hs.load2_at(ho[0] + 128u * k + 16u);
        if (two) {
          hv[1][k].lo = hs.load2_at(ho[1] + 128u * k);
          hv[1][k].hi = hs.load2_at(ho[1] + 128u * k + 16u);
        }
      }
    } else {
      uint32_t xo_next[MT];
      x_offsets(nst ? nst : st, nst != nullptr, xo_next);
      // 1. input part; one weight fragment serves both tiles.  The next
      // step's input fragments are requested during its first half and the
      // child-state fragments of tile 0's rows during its second half, one
      // load or one block per MFMA step, rather than in bursts,
      // which would hold the MFMAs behind them until the address unit has
      // taken every load.  The child fragments are not requested at the
      // start: a level's children are written at the end of the previous
      // level, about when this step begins, so pairs read at once would
      // mostly still carry old tags.
      const float *bx = &Wx_s[i16 * LDX + xcol + 4 * g4];
#pragma unroll
      for (int b = 0; b < NBX; ++b) {
        float4 wv[NTS];
#pragma unroll
        for (int nt = 0; nt < NTS; ++nt) wv[nt] = *(const float4 *)(bx + (NT0 + nt) * 16 * LDX + 16 * b);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          mfma_kstep_xn<NTS>(k, as_float4(xc[0][b]), wv, step_acc(0));
          if (two) mfma_kstep_xn<NTS>(k, as_float4(xc[1][b]), wv, step_acc(1));
          if (b == 0) {
            static_assert(MT * NBX == 4, "one next-step input load per MFMA step");
            xn[k / NBX][k % NBX] = xin.load4(xo_next[k / NBX] + 64u * (k % NBX));
          }
          if (b == NBX - 1) {
            // (tile 1's blocks follow during tile 0's recurrent part)
            static_assert(NBR == 4, "one child block per MFMA step");
            hv[0][k].lo = hs.load2_at(ho[0] + 128u * k);
            hv[0][k].hi = hs.load2_at(ho[0] + 128u * k + 16u);
          }
        }
      }
    }
    CORTEX_TRACE_POINT(l, 1);
    // 2. per tile: wait until its child fragments carry the launch tag, then
    // contract them.  With the fused input part, tile 1's fragments are
    // requested between the MFMA blocks of tile 0's contraction, so the
    // address unit takes half the fragments during the input part and half
    // in the shadow of tile 0's recurrent MFMAs.
    auto wait_tile = [&](int t) __attribute__((always_inline)) {
      auto ready_t = [&]() __attribute__((always_inline)) -> bool {
        bool rt = true;
#pragma unroll
        for (int b = 0; b < NBR; ++b) rt = rt && hv[t][b].ready(tag);
        return cr[t] < 0 || rt;
      };
      if (gave_up || ready_t()) return;
      const uint64_t t0 = wall_clock64();
      for (;;) {
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int b = 0; b < NBR; ++b)
          if (cr[t] >= 0 && !hv[t][b].ready(tag)) {
            hv[t][b].lo = hs.load2_at(ho[t] + 128u * b);
            hv[t][b].hi = hs.load2_at(ho[t] + 128u * b + 16u);
          }
        // the status first: a load still in flight at the exit would hold
        // back the MFMAs that follow until it returns
        if (load_status(a.status) != 0) {
          gave_up = 1;
          break;
        }
        if (ready_t()) break;
        if (wall_clock64() - t0 > a.timeout) {
          raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
          gave_up = 1;
          break;
        }
      }
      if (gave_up) stop_s = 1;             // read by every wave after the next barrier
    };
    wait_tile(0);
    CORTEX_TRACE_POINT(l, 2);
    // 3. recurrent part
#pragma unroll
    for (int b = 0; b < NBR; ++b) {
      mfma_k16_xn<NTS>(hv[0][b].value(true), step_wr(b), step_acc(0));
      if (!kHoisted && two) {
        hv[1][b].lo = hs.load2_at(ho[1] + 128u * b);
        hv[1][b].hi = hs.load2_at(ho[1] + 128u * b + 16u);
      }
    }
    if (two) {
      wait_tile(1);
#pragma unroll
      for (int b = 0; b < NBR; ++b) mfma_k16_xn<NTS>(hv[1][b].value(true), step_wr(b), step_acc(1));
    }
    CORTEX_TRACE_WAVE(l);
    // the next step's input fragments are complete before this step's stores
    // are issued, so its first contraction does not wait for the stores
    if constexpr (!kHoisted)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int b = 0; b < NBX; ++b) settle(xn[t][b]);
#pragma unroll
    for (int t = 0; t < MT; ++t)
      if (t == 0 || two)
#pragma unroll
        for (int nt = NT0; nt < NT0 + NTS; ++nt) {
          const int c = nt * 16 + i16;
          *(floatx4 *)&C_s[((wave * MT + t) * J + c) * kTileM + 4 * (g4 ^ ((c >> 2) & 3))] = acc[t][nt];
        }
    __syncthreads();
    CORTEX_TRACE_POINT(l, 3);
    if (stop_s) return true;               // a wave gave up its wait: every wave stops here
    // epilogue: thread (unit ej, row quarter eq of tile et) sums the eight
    // partial sums of four rows, bias first, and writes them; every output of
    // the thread first, then the stores (a store's data registers are not
    // reused while earlier stores are in flight)
    static_assert(EPI == 4 && kFwdThreads == J * MT * 4, "one row quarter of one tile per thread");
    floatx4 sum = kHoisted ? floatx4{pv[0], pv[1], pv[2], pv[3]} : floatx4{bias_s[ej], bias_s[ej], bias_s[ej], bias_s[ej]};
    if (elive) {
#pragma unroll
      for (int w = 0; w < kFwdWaves; ++w) {
        const floatx4 p = *(const floatx4 *)&C_s[((w * MT + et) * J + ej) * kTileM + 4 * (eq ^ ((ej >> 2) & 3))];
#pragma unroll
        for (int v = 0; v < 4; ++v) sum[v] += p[v];
      }
    }
    // C_s is written again by the next step: every wave has read it once all
    // pass here, before the tanh and the stores, so the stores hold nobody up
    __syncthreads();
    float hv_out[EPI];
    uint32_t el[EPI];
#pragma unroll
    for (int v = 0; v < EPI; ++v) {
      const int row = st[2 + et] + 4 * eq + v;
      hv_out[v] = tanh_f(sum[v]);
      el[v] = (elive && row < lend) ? (uint32_t)(row * H + hbase + ej) : 0xFFFFFFFFu;
    }
    // the tagged pairs (what the next level waits for) first, then the outputs
#pragma unroll
    for (int v = 0; v < EPI; ++v)
      if (el[v] != 0xFFFFFFFFu) hs.store1(el[v], hv_out[v], tag);
#pragma unroll
    for (int v = 0; v < EPI; ++v)
      if (el[v] != 0xFFFFFFFFu) a.h[el[v]] = hv_out[v];
    CORTEX_TRACE_POINT(l, 4);
    return false;
  };

  u32x4 xa[MT][NBX], xb[MT][NBX];
  // one flat pass over this group's steps, level after level, a listed chunk
  // at a time
  auto step = [&](int e) __attribute__((always_inline)) -> const int * { return &list[e * SI]; };
  for (int first = 0;;) {
    // two steps per iteration, written out, so each step's input fragments
    // stay in fixed registers (xa, xb) rather than being selected at run time
    if (!kHoisted && listed > 0) {
      issue_x(step(0), xa, true);
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int b = 0; b < NBX; ++b) settle(xa[t][b]);
    }
    // Steps of one kind (whole or half) run in a loop of their own, entered
    // with no load in flight: a loop entered with another kind's loads
    // pending would wait for them on every iteration, since the compiler's
    // wait counts merge every path into the loop.
    int e = 0;
    auto run_kind = [&](auto half_c) __attribute__((always_inline)) -> bool {
      constexpr int kKind = decltype(half_c)::value;
      for (;;) {
        CORTEX_TRACE_POINT(step(e)[0], 0);
        if (run_step(half_c, step(e), xa, e + 1 < listed ? step(e + 1) : nullptr, xb)) return true;
        CORTEX_TRACE_POINT(step(e)[0], 5);
        if (++e >= listed) return false;
        if (step(e)[5] != kKind) {
          // the next step's input fragments are in xb; the next run reads xa
#pragma unroll
          for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int b = 0; b < NBX; ++b) xa[t][b] = xb[t][b];
          return false;
        }
        CORTEX_TRACE_POINT(step(e)[0], 0);
        if (run_step(half_c, step(e), xb, e + 1 < listed ? step(e + 1) : nullptr, xa)) return true;
        CORTEX_TRACE_POINT(step(e)[0], 5);
        if (++e >= listed || step(e)[5] != kKind) return false;
      }
    };
    while (e < listed) {
      __builtin_amdgcn_s_waitcnt(kWaitVmcntZero);
      const int kind = step(e)[5];
      const bool stop = kind == 1   ? run_kind(std::integral_constant<int, 1>{})
                        : kind == 2 ? run_kind(std::integral_constant<int, 2>{})
                                    : run_kind(std::integral_constant<int, 0>{});
      if (stop) return;
    }
    first += kDagStepCap;
    if (first >= total) break;
    // the next chunk: every wave is done with this one's records
    __syncthreads();
    int bad_chunk = 0;
    list_steps(first, bad_chunk);
    listed = min(total - first, kDagStepCap);
    __syncthreads();                           // the step records are written
    int crow[kFillPer], cv[kFillPer], c0[kFillPer], c1[kFillPer];
#pragma unroll
    for (int k = 0; k < kFillPer; ++k) {
      const int idx = tid + k * kFwdThreads;
      crow[k] = idx < listed * kDagStepRows ? dag_slot_row(&list[(idx / kDagStepRows) * SI], idx % kDagStepRows) : -1;
      cv[k] = c0[k] = c1[k] = -1;
      if (crow[k] >= 0) {
        cv[k] = a.level_nodes[crow[k]];
        c0[k] = a.child_rows[(size_t)crow[k] * 2];
        c1[k] = a.child_rows[(size_t)crow[k] * 2 + 1];
      }
    }
#pragma unroll
    for (int k = 0; k < kFillPer; ++k) {
      const int idx = tid + k * kFwdThreads;
      if (idx < listed * kDagStepRows &&
          !dag_store_codes(a, &list[(idx / kDagStepRows) * SI], idx % kDagStepRows, crow[k] >= 0, cv[k], c0[k], c1[k]))
        bad_chunk = 1;
    }
    if (__syncthreads_or(bad_chunk)) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
  }
  CORTEX_TRACE_KERNEL(3);
  if (a.retire) retire_tag(a.sync, tag, a.status, a.timeout);
}

// ---------------------------------------------------------------------------
// Child-sum TreeLSTM.  Per tile of 16 nodes: the node part x W^T (k split
// over waves 0-3) and the edge part h_k U^T for the 16 x 4 child slots (edge
// tile m = wave & 3, k half = wave >> 2).  The gates are then
//   i, o, u = s(W x + sum_k U h_k + b),  f_k = s(W_f x + U_f h_k + b_f),
//   c = i*u + sum_k f_k * c_k,  h = o * tanh(c)
// (U h~ is taken as sum_k U h_k: the same sum in another order; an absent
// slot reads zero rows, so it adds exactly zero).  Child states come from the
// tagged staging as in the kernel above.
// ---------------------------------------------------------------------------
template <int H, bool kCached, bool kFused = false>
__global__ void __launch_bounds__(kFwdThreads) childsum_forward_kernel(FwdArgs a) {
  constexpr int J = 4;
  using D = Dims<CORTEX_CHILDSUM_TREELSTM, H, J>;
  constexpr int LDW = D::LDW, NBX = D::NBX, NBE = D::NBE, KWX = D::KWX, KWE = D::KWE;
  constexpr int ZW = 7 * J;                 // per row: i, o, u, then f_k * c_k for 4 slots
  // The next tile's operands are requested during the current tile while two
  // operand sets fit the registers; at H = 512 one set (the 16 x 4 child-slot
  // rows alone take 128 VGPRs as tagged pairs) is loaded per tile instead.
  constexpr bool kPrefetch = H <= 256;
  static_assert(D::MPAD == 16 && kTileM * ZW <= kFwdThreads, "one n-tile, one gate item per thread");

  __shared__ __attribute__((aligned(16))) float W_s[16 * LDW];
  __shared__ __attribute__((aligned(16))) float Cx[4 * 16 * 16];     // [4 waves][16 nodes][16]
  __shared__ __attribute__((aligned(16))) float Ce[2 * 64 * 16];     // [2 halves][64 edges][16]
  __shared__ float Z_s[kTileM * ZW];
  __shared__ float bias_s[16];
  __shared__ ChunkRows chunk;
  extern __shared__ int cache[];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  // node group q's slices are workgroups q, q + Q, q + 2Q, ..., which
  // round-robin dispatch puts on the XCDs congruent to q modulo gcd(Q, 8)
  // (two XCDs for Q = 4) instead of spreading a group over all eight
  const int slice = blockIdx.x / a.Q, group = blockIdx.x % a.Q, Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N, K = a.K;
  const uint32_t tag = launch_tag(a.sync);     // read with the status: one round trip
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const TagBuf cs(a.cs, (uint32_t)N * H * 8);
  const InBuf xin(a.x_table, (uint32_t)a.x_rows * H * 4);
  const int em = wave & 3, ehalf = wave >> 2;           // edge m-tile and k half of this wave
  const int e_node = (16 * em + i16) >> 2, e_slot = (16 * em + i16) & 3;
  const int ek = ehalf * KWE + 4 * g4;                  // this lane's edge column in block 0 (16 per block)
  // gate item of this thread: row zi, slot zk (0..2 = i, o, u; 3.. = forget of child zk-3), unit zj
  const int zi = tid / ZW, zk = (tid % ZW) / J, zj = tid % J;

  CORTEX_TRACE_KERNEL(0);
  const int status0 = load_status(a.status);    // one round trip with the weight loads
  Structure<kCached> st;
  int L;
  if constexpr (kFused) {
    static_assert(kCached, "fused launches cache the structure");
    WeightRegs<CORTEX_CHILDSUM_TREELSTM, H, J> wr;
    issue_weight_slice<CORTEX_CHILDSUM_TREELSTM, H, J>(a, hbase, wr);
    const bool ok = fused_structure(a, cache, st, L);
    commit_weight_slice<CORTEX_CHILDSUM_TREELSTM, H, J>(wr, W_s, bias_s);
    if (!ok || status0 != 0) return;
    __syncthreads();                  // the weight slice is in LDS before any tile reads it
    CORTEX_TRACE_KERNEL(1);
  } else {
    load_weight_slice<CORTEX_CHILDSUM_TREELSTM, H, J>(a, hbase, W_s, bias_s);
    if (status0 != 0) return;
    CORTEX_TRACE_KERNEL(1);
    if (!setup_structure<kCached, true, false>(a, cache, st, L)) return;
  }
  CORTEX_TRACE_KERNEL(2);
  if (!mark_entered(a.sync, tag, a.status)) return;
  int gave_up = 0;

  struct TileOps {
    u32x4 xv[NBX];
    Frag ev[NBE];
    int ecr;
    u32x2 cc;
    int ce;
  };

  // ---- level 0: a leaf has no child, so its cell is the node-input part
  //      alone: c = i*u, h = o*tanh(c).  Each of LW waves takes H / LW input
  //      columns, and the input rows of up to kLeafBatch of this group's leaf
  //      tiles (u = group, group + Q, ...) are requested at once, so the
  //      gathers from the input table share one memory round trip ----
  if (a.level_lo == 0) {
    constexpr int LW = (H / 16 < kFwdWaves) ? H / 16 : kFwdWaves;   // waves with input columns
    constexpr int NBL = H / 16 / LW;                                 // 16-blocks per wave
    constexpr int kLeafBatch = 8;
    CORTEX_TRACE_POINT(0, 0);
    const int lr1 = st.offset(L > 1 ? 1 : L);
    if (lr1 < 0 || lr1 > N) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int nt0 = (lr1 + kTileM - 1) / kTileM;
    const int kcol = wave * 16 * NBL + 4 * g4;           // this lane's first input column
    for (int ub = group; ub < nt0; ub += Q * kLeafBatch) {
      u32x4 xl[kLeafBatch][NBL];
#pragma unroll
      for (int k = 0; k < kLeafBatch; ++k) {
        const int row = (ub + k * Q) * kTileM + i16;
        int xr = -1;
        if (wave < LW && ub + k * Q < nt0 && row < lr1) {
          if (kCached) {
            xr = st.input_row(row);
          } else {
            const int v = a.level_nodes[row];
            if (v < 0 || v >= N) {
              raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
            } else {
              xr = a.x_index[v];
              if (xr < -1 || xr >= a.x_rows) {
                raise_status(a.status, CORTEX_ST_INPUT_RANGE);
                xr = -1;
              }
            }
          }
        }
#pragma unroll
        for (int b = 0; b < NBL; ++b)
          xl[k][b] = xin.load4(xr >= 0 ? (uint32_t)((xr * H + kcol + 16 * b) * 4) : kNoSource);
      }
#pragma unroll
      for (int k = 0; k < kLeafBatch; ++k) {
        const int rowbase = (ub + k * Q) * kTileM;
        if (rowbase >= lr1) break;
        if (wave < LW) {
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int b = 0; b < NBL; ++b)
            acc = mfma_k16(as_float4(xl[k][b]), *(const float4 *)&W_s[i16 * LDW + kcol + 16 * b], acc);
#pragma unroll
          for (int v = 0; v < 4; ++v) Ce[(wave * 16 + 4 * g4 + v) * 16 + i16] = acc[v];
        }
        __syncthreads();
        if (tid < kTileM * 16) {           // gate row m = (gate i, o, u or f; unit)
          const int i = tid >> 4, m = tid & 15;
          float sum = bias_s[m];
#pragma unroll
          for (int w = 0; w < LW; ++w) sum += Ce[(w * 16 + i) * 16 + m];
          Z_s[tid] = m / J == 2 ? tanh_f(sum) : sigmoidf(sum);
        }
        __syncthreads();
        if (tid < kTileM * J) {
          const int i = tid / J, j = tid % J, row = rowbase + i;
          if (row < lr1) {
            const float *z = &Z_s[i * 16];
            const float cn = z[j] * z[2 * J + j];
            const float hv = z[J + j] * tanh_f(cn);
            const uint32_t el = (uint32_t)(row * H + hbase + j);
            cs.store1(el, cn, tag);
            hs.store1(el, hv, tag);
            a.c[el] = cn;
            a.h[el] = hv;
          }
        }
        __syncthreads();
      }
    }
    CORTEX_TRACE_POINT(0, 5);
    if (L > 1 && a.level_hi > 1 && a.level_barrier && !grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout))
      return;
  }

  for (int l = a.level_lo > 1 ? a.level_lo : 1; l < L && l < a.level_hi; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = st.offset(l), r1 = st.offset(l + 1);
    if (!kCached && (r1 < r0 || r1 > N || (l == 0 && r0 != 0))) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int ntile = (r1 - r0 + kTileM - 1) / kTileM;
    int u0 = ((group - l) % Q + Q) % Q;

    auto child = [&](int u, int i, int s) __attribute__((always_inline)) -> int {
      const int row = r0 + u * kTileM + i;
      if (row >= r1 || s >= K) return -1;
      if (kCached) return st.child(row, s);
      return chunk.crow[(u - u0) / Q][i][s];
    };
    auto xrow_of = [&](int u, int i) __attribute__((always_inline)) -> int {
      if (kCached) return st.input_row(r0 + u * kTileM + i);
      return chunk.xrow[(u - u0) / Q][i];
    };
    // x fragments (waves 0-3), edge fragments, the child cell of the
    // forget-gate item; absent sources read zeros
    auto issue = [&](int u, TileOps &t) __attribute__((always_inline)) {
      const int row = r0 + u * kTileM + i16;
      int xr = -1;
      if (wave < 4 && row < r1) xr = xrow_of(u, i16);
#pragma unroll
      for (int b = 0; b < NBX; ++b)
        t.xv[b] = xin.load4(xr >= 0 ? (uint32_t)((xr * H + wave * KWX + 16 * b + 4 * g4) * 4) : kNoSource);
      t.ecr = child(u, e_node, e_slot);
      if (t.ecr >= 0) {
#pragma unroll
        for (int b = 0; b < NBE; ++b) {
          const uint32_t so = (uint32_t)(t.ecr * H + ek + 16 * b) * 8u;
          t.ev[b].lo = hs.load2_at(so);
          t.ev[b].hi = hs.load2_at(so + 16u);
        }
      } else {
#pragma unroll
        for (int b = 0; b < NBE; ++b) t.ev[b].lo = t.ev[b].hi = u32x4{0u, 0u, 0u, 0u};
      }
      const int cr = (tid < kTileM * ZW && zk >= 3) ? child(u, zi, zk - 3) : -1;
      t.ce = cr >= 0 ? cr * H + hbase + zj : -1;
      t.cc = cs.load1_at(t.ce >= 0 ? (uint32_t)t.ce * 8u : kNoSource);
    };
    auto all_ready = [&](const TileOps &t) __attribute__((always_inline)) -> bool {
      bool r = t.ce < 0 || t.cc.y == tag;
      if (t.ecr >= 0) {
#pragma unroll
        for (int b = 0; b < NBE; ++b) r = r && t.ev[b].ready(tag);
      }
      return r;
    };

    auto process = [&](int u, TileOps &t, bool more, TileOps &tn) __attribute__((always_inline)) {
      // node-input part first: it needs no child
      floatx4 xacc0 = {0.f, 0.f, 0.f, 0.f}, xacc1 = {0.f, 0.f, 0.f, 0.f};
      if (wave < 4) {
        const float *brow = &W_s[i16 * LDW + wave * KWX + 4 * g4];
#pragma unroll
        for (int b = 0; b < NBX; ++b) {
          const float4 bv = *(const float4 *)(brow + 16 * b);
          if (b & 1) xacc1 = mfma_k16(as_float4(t.xv[b]), bv, xacc1);
          else xacc0 = mfma_k16(as_float4(t.xv[b]), bv, xacc0);
        }
      }
      CORTEX_TRACE_POINT(l, 1);
      if (!gave_up && !all_ready(t)) {
        const uint64_t t0 = wall_clock64();
        for (;;) {
          __builtin_amdgcn_s_sleep(1);
          if (t.ecr >= 0) {
#pragma unroll
            for (int b = 0; b < NBE; ++b)
              if (!t.ev[b].ready(tag)) {
                const uint32_t so = (uint32_t)(t.ecr * H + ek + 16 * b) * 8u;
                t.ev[b].lo = hs.load2_at(so);
                t.ev[b].hi = hs.load2_at(so + 16u);
              }
          }
          if (t.ce >= 0 && t.cc.y != tag) t.cc = cs.load1_at((uint32_t)t.ce * 8u);
          const int stv = load_status(a.status);
          if (all_ready(t)) break;
          if (stv != 0) {
            gave_up = 1;
            break;
          }
          if (wall_clock64() - t0 > a.timeout) {
            raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
            gave_up = 1;
            break;
          }
        }
      }
      CORTEX_TRACE_POINT(l, 2);
      if (more) issue(u + Q, tn);
      floatx4 eacc0 = {0.f, 0.f, 0.f, 0.f}, eacc1 = {0.f, 0.f, 0.f, 0.f};
      if (__ballot(t.ecr >= 0) != 0) {      // skip edge tiles with no child at all (leaves)
        const float *brow = &W_s[i16 * LDW + H + ek];
#pragma unroll
        for (int b = 0; b < NBE; ++b) {
          const float4 bv = *(const float4 *)(brow + 16 * b);
          if (b & 1) eacc1 = mfma_k16(t.ev[b].value(true), bv, eacc1);
          else eacc0 = mfma_k16(t.ev[b].value(true), bv, eacc0);
        }
      }
      CORTEX_TRACE_WAVE(l);
      // the next tile's loads stay in flight through this tile's epilogue
      if (wave < 4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) Cx[(wave * 16 + 4 * g4 + v) * 16 + i16] = xacc0[v] + xacc1[v];
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) Ce[(ehalf * 64 + 16 * em + 4 * g4 + v) * 16 + i16] = eacc0[v] + eacc1[v];
      __syncthreads();
      CORTEX_TRACE_POINT(l, 3);
      // ---- gate items: i, o, u of each (row, unit), and f_k * c_k of each
      //      child slot, one per thread ----
      if (tid < kTileM * ZW) {
        const int gs = zk < 3 ? zk : 3, m = gs * J + zj;
        float sum = bias_s[m] + Cx[(0 * 16 + zi) * 16 + m] + Cx[(1 * 16 + zi) * 16 + m] +
                    Cx[(2 * 16 + zi) * 16 + m] + Cx[(3 * 16 + zi) * 16 + m];
        float zv;
        if (zk < 3) {
#pragma unroll
          for (int s = 0; s < 4; ++s)
            sum += Ce[(0 * 64 + zi * 4 + s) * 16 + m] + Ce[(1 * 64 + zi * 4 + s) * 16 + m];
          zv = zk == 2 ? tanh_f(sum) : sigmoidf(sum);
        } else {
          const int s = zk - 3;
          sum += Ce[(0 * 64 + zi * 4 + s) * 16 + m] + Ce[(1 * 64 + zi * 4 + s) * 16 + m];
          zv = t.ce >= 0 ? sigmoidf(sum) * as_float(t.cc.x) : 0.f;
        }
        Z_s[tid] = zv;
      }
      __syncthreads();
      if (tid < kTileM * J) {
        const int i = tid / J, j = tid % J, row = r0 + u * kTileM + i;
        if (row < r1) {
          const float *z = &Z_s[i * ZW];
          const float cn = z[j] * z[2 * J + j] + ((z[3 * J + j] + z[4 * J + j]) + (z[5 * J + j] + z[6 * J + j]));
          const float hv = z[J + j] * tanh_f(cn);
          const uint32_t el = (uint32_t)(row * H + hbase + j);
          cs.store1(el, cn, tag);
          hs.store1(el, hv, tag);
          a.c[el] = cn;
          a.h[el] = hv;
        }
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 4);
    };

    TileOps ta, tb;
    for (; u0 < ntile; u0 += Q * kChunkTiles) {
      const int u_last = min(ntile - 1, u0 + Q * (kChunkTiles - 1));
      if (!kCached) {
        __syncthreads();
        stage_chunk(a, chunk, u0, (u_last - u0) / Q + 1, Q, r0, r1);
        __syncthreads();
      }
      if constexpr (kPrefetch) {
        issue(u0, ta);
        CORTEX_TRACE_POINT(l, 6);
        for (int u = u0;;) {
          bool more = u + Q <= u_last;
          process(u, ta, more, tb);
          u += Q;
          if (!more) break;
          more = u + Q <= u_last;
          process(u, tb, more, ta);
          u += Q;
          if (!more) break;
        }
      } else {
        for (int u = u0; u <= u_last; u += Q) {
          issue(u, ta);
          CORTEX_TRACE_POINT(l, 6);
          process(u, ta, false, ta);
        }
      }
    }
    CORTEX_TRACE_POINT(l, 5);
    if (__syncthreads_or(gave_up)) return;
    if (a.level_barrier && !grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout)) return;
  }
  CORTEX_TRACE_KERNEL(3);
  if (a.retire) retire_tag(a.sync, tag, a.status, a.timeout);
}

// ---------------------------------------------------------------------------
// TreeRNN at H = 64, unrolled recursion (Secs. 3.1, 7.4): every tree of the
// batch is evaluated by one workgroup from its leaves to its root, so a node
// is computed right after its children on the same compute unit and reads
// their states from LDS; no state crosses workgroups and no workgroup waits
// on another.  Every workgroup derives the same assignment from the
// linearization: parents from the child rows, the root of every row by
// pointer jumping (a child row lies in a strictly lower level, so parent
// rows strictly increase and the jumps end), and the tree of root row t to
// workgroup floor(G * hash(t) / 2^32).  A node with several parents joins
// trees, so such a batch goes whole to workgroup 0.  A workgroup groups its
// own rows by level (a slot per row from a per-level counter; the order
// inside a level does not matter, rows being independent) and walks them
// level by level with one workgroup barrier between levels, as the
// single-workgroup kernel does; weights, tiles and epilogue are the same.
// A workgroup that owns more than kForestStateRows rows keeps its states in
// the output rows instead of LDS (its own stores, ordered by the barriers).
// ---------------------------------------------------------------------------
constexpr int kForestMaxRows = 2048;          // batch limit (per-row arrays in LDS)
constexpr int kForestStateRows = 256;         // owned rows whose states stay in LDS
constexpr int kForestRowsPerThread = kForestMaxRows / kFwdThreads;

// LDS of the forest kernel: the states, then off [N + 1], crow [2N], loc, jp,
// lrow, lx [N], loff [N + 1] and lc [2 kForestStateRows]: 8N + 2 + 512 ints.
static size_t forest_lds_bytes(int32_t N) {
  return (size_t)kForestStateRows * kLdsHStride * sizeof(float) +
         ((size_t)(N + 1) + 2 * (size_t)N + 4 * (size_t)N + (N + 1) + 2 * kForestStateRows) * sizeof(int);
}

// The level walk over a workgroup's own rows lrow[0 .. n), grouped by level
// (level l is lrow[loff[l] .. loff[l+1])); lx[k] is the input row of own
// leaf k.  kLdsState: state k is h_s row k and lc holds the local indices of
// its child slots; otherwise the states are the output rows and the child
// slots are read as rows from crow.
template <bool kLdsState>
__device__ __forceinline__ void forest_levels(const FwdArgs &a, const int *crow, const int *lrow, const int *lc,
                                              const int *lx, const int *loff, int L, float *h_s, const float4 *wr,
                                              const float *bias_s, float (*C_s)[kTileM][kLdsH + 4]) {
  constexpr int H = kLdsH, LDH = kLdsHStride, NB = H / 16;
  constexpr int EPI = kTileM * H / kFwdThreads;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int nt = wave & 3, kh = wave >> 2;
  auto state = [&](int k) __attribute__((always_inline)) -> float * {
    return kLdsState ? h_s + (size_t)k * LDH : a.h + (size_t)lrow[k] * H;
  };
  auto child_state = [&](int c) __attribute__((always_inline)) -> const float * {
    return kLdsState ? h_s + (size_t)c * LDH : a.h + (size_t)c * H;
  };
  // level 0: the leaves are their input rows (zeros without one)
  CORTEX_TRACE_POINT(0, 0);
  for (int e = tid; e < loff[1] * (H / 4); e += kFwdThreads) {
    const int k = e / (H / 4), c4 = e % (H / 4);
    const int xr = lx[k];
    const float4 v = xr >= 0 ? *(const float4 *)&a.x_table[(size_t)xr * H + 4 * c4] : make_float4(0.f, 0.f, 0.f, 0.f);
    *(float4 *)(state(k) + 4 * c4) = v;
  }
  __syncthreads();
  CORTEX_TRACE_POINT(0, 5);
  for (int l = 1; l < L; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int k0 = loff[l], k1 = loff[l + 1];
    for (int kb = k0; kb < k1; kb += kTileM) {
      const int k = kb + i16;
      const int cr = k >= k1 ? -1 : (kLdsState ? lc[2 * k + kh] : crow[2 * lrow[k] + kh]);
      float4 av[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        av[b] = cr >= 0 ? *(const float4 *)(child_state(cr) + 16 * b + 4 * g4) : make_float4(0.f, 0.f, 0.f, 0.f);
      floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (b & 1) acc1 = mfma_k16(av[b], wr[b], acc1);
        else acc0 = mfma_k16(av[b], wr[b], acc0);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) C_s[kh][4 * g4 + v][16 * nt + i16] = acc0[v] + acc1[v];
      __syncthreads();
#pragma unroll
      for (int e = 0; e < EPI; ++e) {
        const int p = tid + e * kFwdThreads, i = p / H, j = p % H;
        if (kb + i < k1) state(kb + i)[j] = tanh_f(bias_s[j] + C_s[0][i][j] + C_s[1][i][j]);
      }
      __syncthreads();
    }
    CORTEX_TRACE_POINT(l, 5);
  }
}

__global__ void __launch_bounds__(kFwdThreads) tree_rnn_forest_kernel(FwdArgs a) {
  constexpr int H = kLdsH, LDH = kLdsHStride, NB = H / 16, RPT = kForestRowsPerThread;
  __shared__ __attribute__((aligned(16))) float C_s[2][kTileM][H + 4];
  __shared__ float bias_s[H];
  __shared__ int wsum[kFwdWaves + 1];
  extern __shared__ __attribute__((aligned(16))) float dyn_s[];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int nt = wave & 3, kh = wave >> 2;
  const int N = a.N, G = gridDim.x, me = blockIdx.x;
  float *h_s = dyn_s;
  int *off = (int *)(dyn_s + (size_t)kForestStateRows * LDH);
  int *crow = off + N + 1, *loc = crow + 2 * N, *jp = loc + N, *lrow = jp + N, *lx = lrow + N;
  int *loff = lx + N, *lc = loff + N + 1;

  CORTEX_TRACE_KERNEL(0);
  const int status0 = load_status(a.status);
  float4 wr[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
    wr[b] = *(const float4 *)(a.W + (size_t)(16 * nt + i16) * 2 * H + kh * H + 16 * b + 4 * g4);
  if (tid < H) bias_s[tid] = a.b[tid];
  const int L = *a.num_levels;
  if (status0 != 0) return;
  if (L < 1 || L > N || N > kForestMaxRows) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  // the structure, every load issued before the first LDS store (node ids
  // of this thread's rows stay in registers)
  int node[RPT], cv[2 * RPT], ov[RPT + 1];
#pragma unroll
  for (int i = 0; i < RPT; ++i) node[i] = tid + i * kFwdThreads < N ? a.level_nodes[tid + i * kFwdThreads] : -1;
#pragma unroll
  for (int i = 0; i < 2 * RPT; ++i) cv[i] = tid + i * kFwdThreads < 2 * N ? a.child_rows[tid + i * kFwdThreads] : -1;
#pragma unroll
  for (int i = 0; i <= RPT; ++i) ov[i] = tid + i * kFwdThreads <= L ? a.level_offsets[tid + i * kFwdThreads] : 0;
#pragma unroll
  for (int i = 0; i < 2 * RPT; ++i)
    if (tid + i * kFwdThreads < 2 * N) crow[tid + i * kFwdThreads] = cv[i];
#pragma unroll
  for (int i = 0; i <= RPT; ++i)
    if (tid + i * kFwdThreads <= L) off[tid + i * kFwdThreads] = ov[i];
  for (int i = tid; i < N; i += kFwdThreads) loc[i] = -1;
  for (int i = tid; i < L; i += kFwdThreads) loff[i] = 0;
  CORTEX_TRACE_KERNEL(1);
  __syncthreads();
  // validation, levels and parents (several parents: the batch is not a forest)
  int bad = 0, multi = 0;
  for (int l = tid; l < L; l += kFwdThreads)
    if (off[l + 1] < off[l] || (l == 0 && off[0] != 0) || (l == L - 1 && off[L] != N)) bad = 1;
  // level of each row: the last l with off[l] <= r, by a branch-free search
  // whose step count is the same for every row, so the rows of a thread
  // search in lockstep
  int rlev[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) rlev[i] = 0;
  for (int step = 1 << (31 - __builtin_clz(L)); step > 0; step >>= 1) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int t = rlev[i] + step;
      if (t < L && off[t] <= tid + i * kFwdThreads) rlev[i] = t;
    }
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = tid + i * kFwdThreads;
    if (r >= N) continue;
    const int start = off[rlev[i]];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int c = crow[2 * r + s];
      if (c < -1 || c >= start || c >= N) {
        bad = 1;
      } else if (c >= 0) {
        const int old = atomicCAS(&loc[c], -1, r);
        if (old != -1 && old != r) multi = 1;
      }
    }
    if (node[i] < 0 || node[i] >= N) bad = 1;
  }
  // input rows of this thread's leaf rows, requested now and used once the
  // own rows are known
  int xi[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = tid + i * kFwdThreads;
    xi[i] = (r < N && rlev[i] == 0 && node[i] >= 0 && node[i] < N) ? a.x_index[node[i]] : -1;
  }
  if (__syncthreads_or(bad)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  multi = __syncthreads_or(multi);
  // the root of every row, by pointer jumping (two jumps per round)
  for (int r = tid; r < N; r += kFwdThreads) jp[r] = loc[r] < 0 ? r : loc[r];
  __syncthreads();
  for (int round = 0; round < 16; ++round) {
    int changed = 0, j[RPT];
#pragma unroll
    for (int i = 0; i < RPT; ++i) j[i] = tid + i * kFwdThreads < N ? jp[tid + i * kFwdThreads] : 0;
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int jj = jp[jp[j[i]]];
      if (tid + i * kFwdThreads < N && jj != j[i]) {
        jp[tid + i * kFwdThreads] = jj;
        changed = 1;
      }
    }
    if (!__syncthreads_or(changed)) break;
  }
  // own rows: a slot in their level's counter; input rows of own leaves
  int slot[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = tid + i * kFwdThreads;
    slot[i] = -1;
    if (r >= N) continue;
    const uint32_t t = (uint32_t)jp[r] * 2654435761u;
    const int owner = multi ? 0 : (int)(((uint64_t)t * (uint32_t)G) >> 32);
    if (owner != me) continue;
    slot[i] = atomicAdd(&loff[rlev[i]], 1);
  }
  __syncthreads();
  // level starts of the own rows (exclusive scan of the counts)
  int run = 0, tot = 0;
  for (int base = 0; base < L; base += kFwdThreads) {
    const int l = base + tid;
    const int cnt = l < L ? loff[l] : 0;
    const int ex = block_excl_scan(cnt, wsum, &tot);
    if (l < L) loff[l] = run + ex;
    run += tot;
  }
  const int n_own = run;
  if (tid == 0) loff[L] = n_own;
  if (n_own == 0) return;
  __syncthreads();
  int inrange = 1;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = tid + i * kFwdThreads;
    if (slot[i] < 0) continue;
    const int k = loff[rlev[i]] + slot[i];
    lrow[k] = r;
    loc[r] = k;
    if (rlev[i] == 0) {
      if (xi[i] < -1 || xi[i] >= a.x_rows) {
        inrange = 0;
        xi[i] = -1;
      }
      lx[k] = xi[i];
    }
  }
  if (!inrange) raise_status(a.status, CORTEX_ST_INPUT_RANGE);
  __syncthreads();
  CORTEX_TRACE_KERNEL(2);
  if (n_own <= kForestStateRows) {
    // child slots of the own rows as local indices (a child has the owner of its parent)
    for (int e = tid; e < 2 * n_own; e += kFwdThreads) {
      const int c = crow[2 * lrow[e >> 1] + (e & 1)];
      lc[e] = c >= 0 ? loc[c] : -1;
    }
    __syncthreads();
    forest_levels<true>(a, crow, lrow, lc, lx, loff, L, h_s, wr, bias_s, C_s);
    for (int e = tid; e < n_own * (H / 4); e += kFwdThreads) {
      const int k = e / (H / 4), c4 = e % (H / 4);
      *(float4 *)&a.h[(size_t)lrow[k] * H + 4 * c4] = *(const float4 *)&h_s[k * LDH + 4 * c4];
    }
  } else {
    forest_levels<false>(a, crow, lrow, lc, lx, loff, L, h_s, wr, bias_s, C_s);
  }
  CORTEX_TRACE_KERNEL(3);
}

// ---------------------------------------------------------------------------
// Child-sum TreeGRU and SimpleTreeGRU.
//   h~ = sum_k h_k,  z = s(W_z x + U_z h~ + b_z),  r_k = s(W_r x + U_r h_k + b_r),
//   h' = tanh(W_h x + U_h m + b_h) with m = sum_k r_k * h_k,
//   TreeGRU h = z*h~ + (1-z)*h';  SimpleTreeGRU h = (1-z)*h'.
// The candidate needs the whole vector m, and each slice forms m only for its
// own units, so a level has two exchanges: phase A (as in the child-sum
// TreeLSTM kernel: node inputs on waves 0-3, the 16 x 4 child-slot rows on
// all waves) gives z, r_k, m and h~ for the slice's units and publishes m as
// (value, launch tag) pairs; phase B waits for the tile's m rows from every
// slice and contracts them with U_h.  Weight-slice rows are (z, r, h, zero)
// x 4 units; the edge contraction uses the U_z and U_r rows, phase B the U_h
// rows (the other rows' results are unused).  Leaves (no child) have m = 0
// and h~ = 0: a leaf phase evaluates them from their inputs alone.
// ---------------------------------------------------------------------------
template <int H, bool kSimple, bool kCached, bool kFused = false>
__global__ void __launch_bounds__(kFwdThreads) treegru_forward_kernel(FwdArgs a) {
  constexpr int J = 4;
  constexpr int LDW = 2 * H + 4;
  constexpr int KWX = H / 4, NBX = KWX / 16;      // node input part: waves 0-3
  constexpr int KWE = H / 2, NBE = KWE / 16;      // edge part: two k halves
  constexpr int BW = (H / 16 < kFwdWaves) ? H / 16 : kFwdWaves;   // phase B waves
  constexpr int KWB = H / BW, NBB = KWB / 16;
  constexpr int ZW = 6 * J;                       // per row: z, W_h x + b_h, then r_k * h_k and h_k per slot
  static_assert(KWB % 16 == 0 && KWX % 16 == 0 && KWE % 16 == 0 && kTileM * ZW <= kFwdThreads, "tiling");

  __shared__ __attribute__((aligned(16))) float W_s[16 * LDW];
  __shared__ __attribute__((aligned(16))) float Cx[4 * 16 * 16];     // [4 waves][16 nodes][16]
  __shared__ __attribute__((aligned(16))) float Ce[2 * 64 * 16];     // [2 halves][64 edges][16]; phase B: [8][16][16]
  __shared__ float Z_s[kTileM * ZW];
  __shared__ float R_s[kTileM * 4 * J][2];        // per (node, slot, unit): r_k * h_k, h_k
  __shared__ float keep_s[kTileM * J][3];         // per (node, unit): z, W_h x + b_h, h~
  __shared__ float bias_s[16];
  __shared__ ChunkRows chunk;
  extern __shared__ int cache[];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  // (consecutive slices here: the group-interleaved order of the slice and
  // child-sum kernels made this kernel slower, 77.5 against 74.4 us per step
  // on a 10-tree batch)
  const int slice = blockIdx.x % a.S, group = blockIdx.x / a.S, Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N, K = a.K;
  const uint32_t tag = launch_tag(a.sync);     // read with the status: one round trip
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const TagBuf ms(a.cs, (uint32_t)N * H * 8);
  const InBuf xin(a.x_table, (uint32_t)a.x_rows * H * 4);
  const int em = wave & 3, ehalf = wave >> 2;
  const int e_node = (16 * em + i16) >> 2, e_slot = (16 * em + i16) & 3;
  const int ek = ehalf * KWE + 4 * g4;
  const int zi = tid / ZW, zk = (tid % ZW) / J, zj = tid % J;   // epilogue item: row, kind, unit

  CORTEX_TRACE_KERNEL(0);
  const int status0 = load_status(a.status);
  Structure<kCached> st;
  int L;
  bool fused_ok = true;
  {
    // weight slice: row m = g*J + j (g = z, r, h, zero); columns [W | U]
    constexpr int ROW4 = (LDW - 4) / 4, ITEMS = 16 * ROW4, PER = (ITEMS + kFwdThreads - 1) / kFwdThreads;
    float4 v[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads, m = idx / ROW4, c4 = idx % ROW4;
      const int g = m / J, hj = hbase + m % J, sg = c4 / (H / 4), o4 = c4 % (H / 4);
      v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (idx < ITEMS && g < 3) v[k] = *(const float4 *)((sg == 0 ? a.W : a.U) + ((size_t)g * H + hj) * H + o4 * 4);
    }
    const float bv = tid < 16 && tid / J < 3 ? a.b[(tid / J) * H + hbase + tid % J] : 0.f;
    if constexpr (kFused) {
      // the batch is linearized while the weight loads are in flight
      static_assert(kCached, "fused launches cache the structure");
      fused_ok = fused_structure(a, cache, st, L);
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * kFwdThreads;
      if (idx < ITEMS) *(float4 *)&W_s[(idx / ROW4) * LDW + (idx % ROW4) * 4] = v[k];
    }
    if (tid < 16) bias_s[tid] = bv;
  }
  if (!fused_ok || status0 != 0) return;
  CORTEX_TRACE_KERNEL(1);
  if constexpr (kFused) {
    __syncthreads();                  // the weight slice is in LDS before any tile reads it
  } else {
    if (!setup_structure<kCached, true, false>(a, cache, st, L)) return;
  }
  CORTEX_TRACE_KERNEL(2);
  if (!mark_entered(a.sync, tag, a.status)) return;
  int gave_up = 0;

  // ---- level 0: leaves (m = 0, h~ = 0): h = (1 - z) tanh(W_h x + b_h) ----
  if (a.level_lo == 0) {
    constexpr int LW = (H / 16 < kFwdWaves) ? H / 16 : kFwdWaves;
    constexpr int NBL = H / 16 / LW;
    constexpr int kLeafBatch = 8;
    CORTEX_TRACE_POINT(0, 0);
    const int lr1 = st.offset(L > 1 ? 1 : L);
    if (lr1 < 0 || lr1 > N) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int nt0 = (lr1 + kTileM - 1) / kTileM;
    const int kcol = wave * 16 * NBL + 4 * g4;
    for (int ub = group; ub < nt0; ub += Q * kLeafBatch) {
      u32x4 xl[kLeafBatch][NBL];
#pragma unroll
      for (int k = 0; k < kLeafBatch; ++k) {
        const int row = (ub + k * Q) * kTileM + i16;
        int xr = -1;
        if (wave < LW && ub + k * Q < nt0 && row < lr1) {
          if (kCached) {
            xr = st.input_row(row);
          } else {
            const int v = a.level_nodes[row];
            if (v < 0 || v >= N) {
              raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
            } else {
              xr = a.x_index[v];
              if (xr < -1 || xr >= a.x_rows) {
                raise_status(a.status, CORTEX_ST_INPUT_RANGE);
                xr = -1;
              }
            }
          }
        }
#pragma unroll
        for (int b = 0; b < NBL; ++b)
          xl[k][b] = xin.load4(xr >= 0 ? (uint32_t)((xr * H + kcol + 16 * b) * 4) : kNoSource);
      }
#pragma unroll
      for (int k = 0; k < kLeafBatch; ++k) {
        const int rowbase = (ub + k * Q) * kTileM;
        if (rowbase >= lr1) break;
        if (wave < LW) {
          floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int b = 0; b < NBL; ++b)
            acc = mfma_k16(as_float4(xl[k][b]), *(const float4 *)&W_s[i16 * LDW + kcol + 16 * b], acc);
#pragma unroll
          for (int v = 0; v < 4; ++v) Ce[(wave * 16 + 4 * g4 + v) * 16 + i16] = acc[v];
        }
        __syncthreads();
        if (tid < kTileM * J) {
          const int i = tid / J, j = tid % J, row = rowbase + i;
          float sz = bias_s[j], sh = bias_s[2 * J + j];
#pragma unroll
          for (int w = 0; w < LW; ++w) {
            sz += Ce[(w * 16 + i) * 16 + j];
            sh += Ce[(w * 16 + i) * 16 + 2 * J + j];
          }
          if (row < lr1) {
            const float hv = (1.f - sigmoidf(sz)) * tanh_f(sh);
            const uint32_t el = (uint32_t)(row * H + hbase + j);
            hs.store1(el, hv, tag);
            a.h[el] = hv;
          }
        }
        __syncthreads();
      }
    }
    CORTEX_TRACE_POINT(0, 5);
    if (L > 1 && a.level_hi > 1 && a.level_barrier && !grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout))
      return;
  }

  for (int l = a.level_lo > 1 ? a.level_lo : 1; l < L && l < a.level_hi; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = st.offset(l), r1 = st.offset(l + 1);
    if (!kCached && (r1 < r0 || r1 > N)) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int ntile = (r1 - r0 + kTileM - 1) / kTileM;
    // one pass per level; two (phase A of every tile, a device-wide barrier,
    // then phase B) under level_barrier 2
    const int npass = a.level_barrier == 2 ? 2 : 1;
    for (int pass = 0; pass < npass; ++pass) {
    const bool doA = pass == 0, doB = pass == npass - 1;
    if (pass == 1) {
      if (__syncthreads_or(gave_up)) return;
      if (!grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout)) return;
    }
    for (int u0 = ((group - l) % Q + Q) % Q; u0 < ntile; u0 += Q * kChunkTiles) {
      const int u_last = min(ntile - 1, u0 + Q * (kChunkTiles - 1));
      if (!kCached) {
        __syncthreads();
        stage_chunk(a, chunk, u0, (u_last - u0) / Q + 1, Q, r0, r1);
        __syncthreads();
      }
      auto child = [&](int u, int i, int s) __attribute__((always_inline)) -> int {
        const int row = r0 + u * kTileM + i;
        if (row >= r1 || s >= K) return -1;
        if (kCached) return st.child(row, s);
        return chunk.crow[(u - u0) / Q][i][s];
      };
      for (int u = u0; u <= u_last; u += Q) {
        const int rowbase = r0 + u * kTileM;
        const size_t plane = (size_t)N * H;
        if (doA) {
        // ---- phase A operands: node inputs (waves 0-3), child-slot rows, and
        //      this item's child state h_k[unit] ----
        u32x4 xv[NBX];
        {
          int xr = -1;
          if (wave < 4 && rowbase + i16 < r1) xr = kCached ? st.input_row(rowbase + i16) : chunk.xrow[(u - u0) / Q][i16];
#pragma unroll
          for (int b = 0; b < NBX; ++b)
            xv[b] = xin.load4(xr >= 0 ? (uint32_t)((xr * H + wave * KWX + 16 * b + 4 * g4) * 4) : kNoSource);
        }
        const int ecr = child(u, e_node, e_slot);
        Frag ev[NBE];
#pragma unroll
        for (int b = 0; b < NBE; ++b) {
          const uint32_t so = ecr >= 0 ? (uint32_t)(ecr * H + ek + 16 * b) * 8u : kNoSource;
          ev[b].lo = hs.load2_at(so);
          ev[b].hi = hs.load2_at(so + 16u);
        }
        const int icr = (tid < kTileM * ZW && zk >= 2) ? child(u, zi, zk - 2) : -1;
        const int ie = icr >= 0 ? icr * H + hbase + zj : -1;
        u32x2 ih = hs.load1_at(ie >= 0 ? (uint32_t)ie * 8u : kNoSource);
        // node-input part first: it needs no child
        floatx4 xacc0 = {0.f, 0.f, 0.f, 0.f}, xacc1 = {0.f, 0.f, 0.f, 0.f};
        if (wave < 4) {
          const float *brow = &W_s[i16 * LDW + wave * KWX + 4 * g4];
#pragma unroll
          for (int b = 0; b < NBX; ++b) {
            const float4 bv = *(const float4 *)(brow + 16 * b);
            if (b & 1) xacc1 = mfma_k16(as_float4(xv[b]), bv, xacc1);
            else xacc0 = mfma_k16(as_float4(xv[b]), bv, xacc0);
          }
        }
        CORTEX_TRACE_POINT(l, 1);
        auto ready_a = [&]() __attribute__((always_inline)) -> bool {
          bool r = ie < 0 || ih.y == tag;
          if (ecr >= 0) {
#pragma unroll
            for (int b = 0; b < NBE; ++b) r = r && ev[b].ready(tag);
          }
          return r;
        };
        if (!gave_up && !ready_a()) {
          const uint64_t t0 = wall_clock64();
          for (;;) {
            __builtin_amdgcn_s_sleep(1);
            if (ecr >= 0) {
#pragma unroll
              for (int b = 0; b < NBE; ++b)
                if (!ev[b].ready(tag)) {
                  const uint32_t so = (uint32_t)(ecr * H + ek + 16 * b) * 8u;
                  ev[b].lo = hs.load2_at(so);
                  ev[b].hi = hs.load2_at(so + 16u);
                }
            }
            if (ie >= 0 && ih.y != tag) ih = hs.load1_at((uint32_t)ie * 8u);
            const int stv = load_status(a.status);
            if (ready_a()) break;
            if (stv != 0) {
              gave_up = 1;
              break;
            }
            if (wall_clock64() - t0 > a.timeout) {
              raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
              gave_up = 1;
              break;
            }
          }
        }
        CORTEX_TRACE_POINT(l, 2);
        floatx4 eacc0 = {0.f, 0.f, 0.f, 0.f}, eacc1 = {0.f, 0.f, 0.f, 0.f};
        if (__ballot(ecr >= 0) != 0) {
          const float *brow = &W_s[i16 * LDW + H + ek];
#pragma unroll
          for (int b = 0; b < NBE; ++b) {
            const float4 bv = *(const float4 *)(brow + 16 * b);
            if (b & 1) eacc1 = mfma_k16(ev[b].value(true), bv, eacc1);
            else eacc0 = mfma_k16(ev[b].value(true), bv, eacc0);
          }
        }
        if (wave < 4) {
#pragma unroll
          for (int v = 0; v < 4; ++v) Cx[(wave * 16 + 4 * g4 + v) * 16 + i16] = xacc0[v] + xacc1[v];
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) Ce[(ehalf * 64 + 16 * em + 4 * g4 + v) * 16 + i16] = eacc0[v] + eacc1[v];
        __syncthreads();
        // ---- phase A epilogue: z, W_h x + b_h per (node, unit); r_k * h_k
        //      and h_k per (node, slot, unit) ----
        if (tid < kTileM * ZW) {
          const int gz = zk == 0 ? 0 : (zk == 1 ? 2 : 1);      // gate row: z, h or r
          const int m = gz * J + zj;
          float sum = bias_s[m] + Cx[(0 * 16 + zi) * 16 + m] + Cx[(1 * 16 + zi) * 16 + m] +
                      Cx[(2 * 16 + zi) * 16 + m] + Cx[(3 * 16 + zi) * 16 + m];
          if (zk == 0) {                 // z: U_z h~ = sum over the child slots of U_z h_k
#pragma unroll
            for (int s = 0; s < 4; ++s)
              sum += Ce[(0 * 64 + zi * 4 + s) * 16 + m] + Ce[(1 * 64 + zi * 4 + s) * 16 + m];
            Z_s[tid] = sigmoidf(sum);
          } else if (zk == 1) {
            Z_s[tid] = sum;
          } else {
            const int s = zk - 2;
            sum += Ce[(0 * 64 + zi * 4 + s) * 16 + m] + Ce[(1 * 64 + zi * 4 + s) * 16 + m];
            const float hk = ie >= 0 ? as_float(ih.x) : 0.f;
            R_s[(zi * 4 + s) * J + zj][0] = ie >= 0 ? sigmoidf(sum) * hk : 0.f;
            R_s[(zi * 4 + s) * J + zj][1] = hk;
          }
        }
        __syncthreads();
        if (tid < kTileM * J) {
          const int i = tid / J, j = tid % J, row = rowbase + i;
          float mv = 0.f, hsum = 0.f;
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            mv += R_s[(i * 4 + s) * J + j][0];
            hsum += R_s[(i * 4 + s) * J + j][1];
          }
          keep_s[tid][0] = Z_s[i * ZW + j];
          keep_s[tid][1] = Z_s[i * ZW + J + j];
          keep_s[tid][2] = hsum;
          if (row < r1) {
            const uint32_t el = (uint32_t)(row * H + hbase + j);
            ms.store1(el, mv, tag);
            if (!doB) {                  // phase B runs after the barrier: keep z, W_h x + b_h, h~
              a.keep[el] = keep_s[tid][0];
              a.keep[plane + el] = keep_s[tid][1];
              a.keep[2 * plane + el] = hsum;
            }
          }
        }
        }                                // doA
        if (!doB) continue;
        if (!doA && tid < kTileM * J) {  // the same thread wrote them before the barrier
          const int row = rowbase + tid / J;
          if (row < r1) {
            const size_t el = (size_t)row * H + hbase + tid % J;
            keep_s[tid][0] = a.keep[el];
            keep_s[tid][1] = a.keep[plane + el];
            keep_s[tid][2] = a.keep[2 * plane + el];
          }
        }
        // ---- phase B: the tile's m rows from every slice, contracted with U_h ----
        Frag mf[NBB];
        const int mrow = (wave < BW) ? rowbase + i16 : r1;       // waves past BW have no columns
#pragma unroll
        for (int b = 0; b < NBB; ++b) {
          const uint32_t so = mrow < r1 ? (uint32_t)(mrow * H + wave * KWB + 16 * b + 4 * g4) * 8u : kNoSource;
          mf[b].lo = ms.load2_at(so);
          mf[b].hi = ms.load2_at(so + 16u);
        }
        auto ready_b = [&]() __attribute__((always_inline)) -> bool {
          bool r = true;
#pragma unroll
          for (int b = 0; b < NBB; ++b) r = r && mf[b].ready(tag);
          return mrow >= r1 || r;
        };
        if (!gave_up && !ready_b()) {
          const uint64_t t0 = wall_clock64();
          for (;;) {
            __builtin_amdgcn_s_sleep(1);
#pragma unroll
            for (int b = 0; b < NBB; ++b)
              if (!mf[b].ready(tag)) {
                const uint32_t so = (uint32_t)(mrow * H + wave * KWB + 16 * b + 4 * g4) * 8u;
                mf[b].lo = ms.load2_at(so);
                mf[b].hi = ms.load2_at(so + 16u);
              }
            const int stv = load_status(a.status);
            if (ready_b()) break;
            if (stv != 0) {
              gave_up = 1;
              break;
            }
            if (wall_clock64() - t0 > a.timeout) {
              raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
              gave_up = 1;
              break;
            }
          }
        }
        floatx4 bacc = {0.f, 0.f, 0.f, 0.f};
        if (wave < BW) {
          const float *brow = &W_s[i16 * LDW + H + wave * KWB + 4 * g4];
#pragma unroll
          for (int b = 0; b < NBB; ++b) bacc = mfma_k16(mf[b].value(true), *(const float4 *)(brow + 16 * b), bacc);
        }
        __syncthreads();                  // every wave is past its reads of Ce (phase A)
        if (wave < BW) {
#pragma unroll
          for (int v = 0; v < 4; ++v) Ce[(wave * 16 + 4 * g4 + v) * 16 + i16] = bacc[v];
        }
        __syncthreads();
        CORTEX_TRACE_POINT(l, 3);
        if (tid < kTileM * J) {
          const int i = tid / J, j = tid % J, row = rowbase + i;
          float sh = keep_s[tid][1];
#pragma unroll
          for (int w = 0; w < BW; ++w) sh += Ce[(w * 16 + i) * 16 + 2 * J + j];
          const float zv = keep_s[tid][0];
          const float cand = tanh_f(sh);
          const float hv = kSimple ? (1.f - zv) * cand : zv * keep_s[tid][2] + (1.f - zv) * cand;
          if (row < r1) {
            const uint32_t el = (uint32_t)(row * H + hbase + j);
            hs.store1(el, hv, tag);
            a.h[el] = hv;
          }
        }
        __syncthreads();
        CORTEX_TRACE_POINT(l, 4);
      }
    }
    }                                    // pass
    CORTEX_TRACE_POINT(l, 5);
    if (__syncthreads_or(gave_up)) return;
    if (a.level_barrier && !grid_sync<false>(SyncWords{a.sync}, a.status, a.timeout)) return;
  }
  CORTEX_TRACE_KERNEL(3);
  if (a.retire) retire_tag(a.sync, tag, a.status, a.timeout);
}

// Validated level bounds; false (and a status) when the linearization is broken.
__device__ __forceinline__ bool level_bounds(const FwdArgs &a, int l, int &r0, int &r1) {
  r0 = a.level_offsets[l];
  r1 = a.level_offsets[l + 1];
  if (r0 < 0 || r1 < r0 || r1 > a.N || (l == 0 && r0 != 0)) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return false;
  }
  return true;
}

// ---------------------------------------------------------------------------
// MV-RNN (d = 64 or 128): p = tanh(W [B a; A b]), P = W_M [A; B].
// Node-parallel: with RB = d / 16 row blocks and G/RB node groups, workgroup
// b owns output rows [16 r, 16 r + 16), r = b / (G/RB), of every node it
// processes (its 16 rows of W_M in LDS, its share of the same rows of W in
// registers), and node group q = b % (G/RB) takes nodes q, q + G/RB, ... of
// each level.  P = W_M[A;B] runs on MFMA with
// [A;B] staged in LDS (wave w computes output columns 16w .. 16w+15, so a
// workgroup has d/16 waves); the matrix-vector products use VALU.  Levels are
// ordered per datum, as in the slice kernels: every element of p and P is
// also published as a (value, launch tag) pair, a workgroup waits for
// exactly the child vectors and matrices it stages, and a leaf child is read
// from the inputs (its state is the given (a, A)), so nothing waits on the
// leaf level.  Child rows and the input rows of the leaves are cached in LDS
// for batches of up to MvDims<D>::kCacheRows rows.
// ---------------------------------------------------------------------------
template <int D>
struct MvDims {
  static constexpr int kThreads = 4 * D;                 // d/16 waves
  static constexpr int RB = D / 16;                      // row blocks of P per node
  static constexpr int kLd = 2 * D + 4;                  // W_M slice row stride
  static constexpr int kAb = D + 1;                      // [A;B] row stride (odd: row-wise reads spread banks)
  static constexpr int kGroups = 2 * D * D / 4 / kThreads;   // float4 groups of [A;B] per thread
  static constexpr int kSide = D * D / 4;                // float4 groups per matrix
  static constexpr int kParts = kThreads / 16;           // partial sums per output of p (8 terms each)
  // the cache (3 ints per row) must fit beside the static LDS: 36 KB at
  // d = 64, 7.5 KB at d = 128 (where [A;B] alone takes 129 KB)
  static constexpr int kCacheRows = D == 64 ? 3072 : 640;
  static_assert(kParts * 8 == 2 * D && kGroups * kThreads * 4 == 2 * D * D, "MV-RNN tiling");
};
constexpr int kMvD = 64, kMvD2 = 128;

// Fused launches (cortex_tree_infer): the batch is linearized in LDS first.
// Dynamic LDS (ints): child rows (2N), leaf input rows (N), level offsets
// (N + 1), input row by node id (N), then the linearizer's arrays.
template <int D>
constexpr int kMvFusedPer = kFusedMaxNodes / MvDims<D>::kThreads;      // nodes per thread: N <= 2048
template <int D>
__host__ __device__ inline size_t mv_fused_ints(int N) {
  return 5 * (size_t)N + 1 + small_lin_ints<MvDims<D>::kThreads>(N, 2);
}

template <int D, bool kFused = false>
__global__ void __launch_bounds__(MvDims<D>::kThreads) mvrnn_forward_kernel(FwdArgs a) {
  using M = MvDims<D>;
  constexpr int kThreads = M::kThreads, RB = M::RB, kLd = M::kLd, kAb = M::kAb, kGroups = M::kGroups;
  constexpr int kSide = M::kSide, kParts = M::kParts;
  constexpr int WPER = 16 * 2 * D / kThreads;
  __shared__ float WM_s[16 * kLd];
  __shared__ float AB_s[2 * D * kAb];
  __shared__ float vec_s[2 * D];          // a (left vector), b (right vector)
  __shared__ float bab_s[2 * D];          // [B a; A b]
  __shared__ int src_s[2][2];             // per child slot: staged row or -1, input row or -1
  extern __shared__ int mv_cache[];       // cached: child rows [N*2], then leaf input rows [off1]

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  // node group g's RB workgroups are g, g + G/RB, ...: round-robin dispatch
  // puts them on one XCD
  const int ngroups = gridDim.x / RB, rblk = blockIdx.x / ngroups, ngroup = blockIdx.x % ngroups;
  const int N = a.N;
  const bool cached = kFused || N <= M::kCacheRows;
  const uint32_t tag = launch_tag(a.sync);     // read with the status: one round trip
  const TagBuf hs(a.hs, (uint32_t)N * D * 8);
  const TagBuf ps(a.cs, (uint32_t)N * D * D * 8);
  const InBuf xv(a.x_table, a.x_table ? (uint32_t)a.x_rows * D * 4 : 0u);
  const InBuf xm(a.leaf_mat, a.leaf_mat ? (uint32_t)a.x_rows * D * D * 4 : 0u);
  // p: output o of this workgroup's 16, partial sum over columns [8 part, 8 part + 8)
  const int po = tid / kParts, ppart = tid % kParts;

  // status, level count and weights requested together
  const int status0 = load_status(a.status);
  int L = kFused ? 0 : *a.num_levels;
  float wv[8];                            // W[16 rblk + po][8 ppart .. +8], for the whole launch
  {
    float wm[WPER];
#pragma unroll
    for (int k = 0; k < WPER; ++k) {
      const int idx = tid + k * kThreads, r = idx / (2 * D), c = idx % (2 * D);
      wm[k] = a.W_M[(size_t)(rblk * 16 + r) * 2 * D + c];
    }
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) wv[kk] = a.W[(size_t)(rblk * 16 + po) * 2 * D + ppart * 8 + kk];
#pragma unroll
    for (int k = 0; k < WPER; ++k) {
      const int idx = tid + k * kThreads, r = idx / (2 * D), c = idx % (2 * D);
      WM_s[r * kLd + c] = wm[k];
    }
  }
  int *crow_c = mv_cache, *leafx_c = mv_cache + 2 * N, *lvo = mv_cache + 3 * N;
  if constexpr (kFused) {
    // linearize the batch (its loads share the weights' round trip), then
    // child rows, level offsets and the leaves' input rows from LDS
    constexpr int PER = kMvFusedPer<D>;
    int *xnode = lvo + N + 1, *lin = xnode + N;
    int xi[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int v = tid + k * kThreads;
      xi[k] = v < N ? a.x_index[v] : -1;
    }
    SmallLin m;
    L = small_linearize<kThreads, PER>(a.children, N, 2, a.status, lin, m, fused_lin_stamps(a));
    if (L == 0) return;
    if (blockIdx.x == 0)
      small_lin_emit<kThreads>(m, N, 2, L, a.o_num_levels, a.o_height, a.o_level_offsets, a.o_level_nodes,
                               a.o_node_row, a.o_child_rows);
    for (int i = tid; i <= L; i += kThreads) lvo[i] = i < L ? m.lcount[i] : N;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int v = tid + k * kThreads;
      if (v < N) {
        int x = xi[k];
        if (x < -1 || x >= a.x_rows) {
          raise_status(a.status, CORTEX_ST_INPUT_RANGE);
          x = -1;
        }
        xnode[v] = x;
      }
    }
    __syncthreads();
    for (int r = tid; r < N; r += kThreads) {
      const int v = m.order[r];
      leafx_c[r] = xnode[v];
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int c = m.ch[v * 2 + s];
        crow_c[r * 2 + s] = c < 0 ? -1 : m.nrow[c];
      }
    }
    __syncthreads();
  }
  if (status0 != 0) return;
  if (L < 1 || L > N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  if (!mark_entered(a.sync, tag, a.status)) return;
  int r0, r1;
  auto bounds = [&](int l) -> bool {
    if constexpr (kFused) {
      r0 = lvo[l];
      r1 = lvo[l + 1];
      return true;
    } else {
      return level_bounds(a, l, r0, r1);
    }
  };
  if (!bounds(0)) return;
  const int off1 = r1;

  // input row of leaf row r (validated), -1 = none
  auto leaf_input = [&](int r) -> int {
    const int v = a.level_nodes[r];
    if (v < 0 || v >= N) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return -1;
    }
    const int xi = a.x_index[v];
    if (xi < -1 || xi >= a.x_rows) {
      raise_status(a.status, CORTEX_ST_INPUT_RANGE);
      return -1;
    }
    return xi;
  };
  if (cached && !kFused) {
    for (int i = tid; i < 2 * N; i += kThreads) {
      int c = a.child_rows[i];
      if (c < -1 || c >= N) {
        raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
        c = -1;
      }
      crow_c[i] = c;
    }
    for (int r = tid; r < off1; r += kThreads) leafx_c[r] = leaf_input(r);
    __syncthreads();
  }

  // leaves: (p, P) = (x_table[x], leaf_mat[x]) or zeros; rows spread over all
  // workgroups, plain stores (no workgroup reads them back)
  for (int r = blockIdx.x; r < off1; r += gridDim.x) {
    const int xi = cached ? leafx_c[r] : leaf_input(r);
    if (tid < D / 4) {
      const float4 val = as_float4(xv.load4(xi >= 0 ? (uint32_t)((xi * D + tid * 4) * 4) : kNoSource));
      *(float4 *)&a.h[(size_t)r * D + tid * 4] = val;
    }
    for (int e = tid; e < D * D / 4; e += kThreads) {
      const float4 val = as_float4(xm.load4(xi >= 0 ? (uint32_t)((xi * D * D + e * 4) * 4) : kNoSource));
      *(float4 *)&a.c[(size_t)r * D * D + e * 4] = val;
    }
  }

  int gave_up = 0;
  for (int l = 1; l < L && !gave_up; ++l) {
    if (!bounds(l)) return;
    for (int r = r0 + ngroup; r < r1; r += ngroups) {
      if (tid < 2) {
        int cr = cached ? crow_c[r * 2 + tid] : a.child_rows[(size_t)r * 2 + tid];
        if (cr < -1 || cr >= r0) {              // a child must sit in a lower level
          raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
          cr = -1;
        }
        src_s[tid][0] = cr >= off1 ? cr : -1;
        src_s[tid][1] = (cr >= 0 && cr < off1) ? (cached ? leafx_c[cr] : leaf_input(cr)) : -1;
      }
      __syncthreads();
      // [A; B]: float4 group f = tid + k*kThreads is side f / kSide (0 = A
      // from slot 0, 1 = B from slot 1), element 4 (f mod kSide) of that matrix
      u32x4 lo[kGroups], hi[kGroups];
#pragma unroll
      for (int k = 0; k < kGroups; ++k) {
        const int f = tid + k * kThreads, side = f / kSide, e4 = (f % kSide) * 4;
        const int st = src_s[side][0], xi = src_s[side][1];
        if (st >= 0) {
          const uint32_t so = (uint32_t)(st * D * D + e4) * 8u;
          lo[k] = ps.load2_at(so);
          hi[k] = ps.load2_at(so + 16u);
        } else {
          lo[k] = xm.load4(xi >= 0 ? (uint32_t)((xi * D * D + e4) * 4) : kNoSource);
          hi[k] = u32x4{0u, 0u, 0u, 0u};
        }
      }
      // vectors: thread t < 2d takes element t mod d of side t / d
      const int vside = (tid / D) & 1, vk = tid % D;
      const int vst = src_s[vside][0], vxi = src_s[vside][1];
      u32x2 vv = {0u, 0u};
      if (tid < 2 * D) {
        if (vst >= 0) vv = hs.load1_at((uint32_t)(vst * D + vk) * 8u);
        else vv.x = xv.load1(vxi >= 0 ? (uint32_t)((vxi * D + vk) * 4) : kNoSource);
      }
      auto ready = [&]() -> bool {
        bool ok = !(tid < 2 * D && vst >= 0) || vv.y == tag;
#pragma unroll
        for (int k = 0; k < kGroups; ++k) {
          const int side = (tid + k * kThreads) / kSide;
          if (src_s[side][0] >= 0) ok = ok && lo[k].y == tag && lo[k].w == tag && hi[k].y == tag && hi[k].w == tag;
        }
        return ok;
      };
      if (!ready()) {
        const uint64_t t0 = wall_clock64();
        for (;;) {
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int k = 0; k < kGroups; ++k) {
            const int f = tid + k * kThreads, side = f / kSide, st = src_s[side][0];
            if (st >= 0 && !(lo[k].y == tag && lo[k].w == tag && hi[k].y == tag && hi[k].w == tag)) {
              const uint32_t so = (uint32_t)(st * D * D + (f % kSide) * 4) * 8u;
              lo[k] = ps.load2_at(so);
              hi[k] = ps.load2_at(so + 16u);
            }
          }
          if (tid < 2 * D && vst >= 0 && vv.y != tag) vv = hs.load1_at((uint32_t)(vst * D + vk) * 8u);
          const int stv = load_status(a.status);
          if (ready()) break;
          if (stv != 0) {
            gave_up = 1;
            break;
          }
          if (wall_clock64() - t0 > a.timeout) {
            raise_status(a.status, CORTEX_ST_BARRIER_TIMEOUT);
            gave_up = 1;
            break;
          }
        }
      }
#pragma unroll
      for (int k = 0; k < kGroups; ++k) {
        const int f = tid + k * kThreads, side = f / kSide, e4 = (f % kSide) * 4;
        const bool staged = src_s[side][0] >= 0;
        const float4 val = make_float4(as_float(lo[k].x), as_float(staged ? lo[k].z : lo[k].y),
                                       as_float(staged ? hi[k].x : lo[k].z), as_float(staged ? hi[k].z : lo[k].w));
        float *dst = &AB_s[(side * D + e4 / D) * kAb + e4 % D];
        dst[0] = val.x;
        dst[1] = val.y;
        dst[2] = val.z;
        dst[3] = val.w;
      }
      if (tid < 2 * D) vec_s[tid] = as_float(vv.x);
      if (__syncthreads_or(gave_up)) {
        gave_up = 1;
        break;
      }
      // [B a; A b]: thread k<d -> (B a)[k] = sum_n B[k][n] a[n];  k>=d -> (A b)[k-d]
      if (tid < 2 * D) {
        const int k = tid % D;
        const float *mrow = (tid < D) ? &AB_s[(D + k) * kAb] : &AB_s[k * kAb];
        const float *vw = (tid < D) ? &vec_s[0] : &vec_s[D];
        float s = 0.f;
        for (int n2 = 0; n2 < D; ++n2) s += mrow[n2] * vw[n2];
        bab_s[tid] = s;
      }
      // P rows [16*rblk, +16) = W_M[rows] [A;B]: wave w -> output columns 16w..16w+15
      floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
      for (int k0 = 0; k0 < 2 * D; k0 += 8) {
        acc0 = mfma16x16x4(WM_s[i16 * kLd + k0 + g4], AB_s[(k0 + g4) * kAb + wave * 16 + i16], acc0);
        acc1 = mfma16x16x4(WM_s[i16 * kLd + k0 + 4 + g4], AB_s[(k0 + 4 + g4) * kAb + wave * 16 + i16], acc1);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const uint32_t el = (uint32_t)(r * D * D + (rblk * 16 + 4 * g4 + v) * D + wave * 16 + i16);
        const float pv = acc0[v] + acc1[v];
        ps.store1(el, pv, tag);
        a.c[el] = pv;
      }
      __syncthreads();
      // p rows: 16 outputs x kParts partial sums of 8 terms, reduced over
      // kParts consecutive lanes
      {
        float s = 0.f;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) s += wv[kk] * bab_s[ppart * 8 + kk];
        for (int sh = kParts / 2; sh > 0; sh >>= 1) s += __shfl_xor(s, sh, kParts);
        if (ppart == 0) {
          const uint32_t el = (uint32_t)(r * D + rblk * 16 + po);
          const float pv = tanh_f(s);
          hs.store1(el, pv, tag);
          a.h[el] = pv;
        }
      }
      __syncthreads();
    }
  }
  if (a.retire) retire_tag(a.sync, tag, a.status, a.timeout);
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
typedef void (*KernelFn)(FwdArgs);

struct Instance {
  KernelFn fn;
  int J;
  int threads;
  size_t lds = SIZE_MAX;        // dynamic LDS the kernel sizes itself (SIZE_MAX: the structure cache)
  bool level_barrier_ok = false;   // honours FwdArgs.level_barrier
  bool level_range_ok = false;     // honours FwdArgs.level_lo / level_hi
  bool phase_barrier_ok = false;   // has two exchanges per level and honours level_barrier 2
  bool one_group = false;          // the whole batch in one workgroup
  int ablate_bits = 0;             // FwdArgs.ablate bits the kernel honours
};

constexpr size_t kStructCacheBudget = 40 * 1024;    // bytes of LDS for the cached linearization

// ints of the structure cache: offsets (<= N+1), child rows, input rows, node ids
// (child-sum: offsets, child rows, input rows; the slice kernels: offsets,
// source codes, input rows of the leaf-input cells)
static size_t cache_ints(int cell, int32_t N, int32_t K) {
  if (cell == CORTEX_CHILDSUM_TREELSTM || cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU)
    return (size_t)N + 1 + (size_t)N * K + N;
  const size_t segs = cell == CELL_DAG ? 3 : 2;
  return (size_t)N + 1 + (size_t)N * segs + (cell == CELL_DAG ? 0 : N);
}

template <int CELL, int H, int J>
static void pick_slice(bool cached, Instance &out) {
  out.J = J;
  out.threads = kFwdThreads;
  out.level_barrier_ok = out.level_range_ok = true;
  if constexpr (CELL == CORTEX_CHILDSUM_TREELSTM) {
    out.fn = cached ? childsum_forward_kernel<H, true> : childsum_forward_kernel<H, false>;
  } else {
    if (knob(CORTEX_KNOB_ABLATE) & 1)       // the instance without model persistence
      out.fn = cached ? slice_forward_kernel<CELL, H, J, true, true> : slice_forward_kernel<CELL, H, J, false, true>;
    else
      out.fn = cached ? slice_forward_kernel<CELL, H, J, true> : slice_forward_kernel<CELL, H, J, false>;
    out.ablate_bits = SrcCfg<CELL>::kLeafX ? 3 : 1;
  }
}

// units per slice: the knob's value where an instance exists, else the default
static bool pick(int cell, int H, int32_t N, bool cached, Instance &out) {
  const int64_t units = knob(CORTEX_KNOB_FWD_SLICE_UNITS);
  // TreeRNN at H = 64: the whole batch in one workgroup while it fits LDS,
  // then one workgroup per tree, then hidden slices; the unroll knob forces
  // the level-parallel slices (1) or one workgroup per tree (2)
  const int64_t unroll = knob(CORTEX_KNOB_TREE_UNROLL);
  const int64_t groups = knob(CORTEX_KNOB_FWD_NODE_GROUPS);
  if (cell == CORTEX_TREE_RNN && H == kLdsH && unroll == 0 && N <= kLdsMaxRows && groups <= 1) {
    out.fn = tree_rnn_lds_kernel<false>;  // one workgroup, every state in LDS
    out.J = kLdsH;
    out.threads = kFwdThreads;
    out.one_group = true;
    out.lds = (size_t)N * kLdsHStride * sizeof(float) + (4 * (size_t)N + 2) * sizeof(int);
    return true;
  }
  if (cell == CORTEX_TREE_RNN && H == kLdsH && ((unroll == 0 && groups == 0) || unroll == 2)) {
    if (N > kForestMaxRows) {
      if (unroll == 2) return false;
    } else {
      out.fn = tree_rnn_forest_kernel;
      out.J = kLdsH;
      out.threads = kFwdThreads;
      out.lds = forest_lds_bytes(N);
      return true;
    }
  }
  if (cell == CORTEX_NARY_TREELSTM && H == 256 && units == 2) {
    pick_slice<CORTEX_NARY_TREELSTM, 256, 2>(cached, out);
    return true;
  }
  // DAG-RNN at H = 256: four 64-unit slices for large batches (operand
  // re-reads dominate there), sixteen 16-unit slices for small ones (a
  // tile's contraction is 4x shorter, and small levels are latency-bound);
  // the knob forces either (16 or 64)
  if (cell == CELL_DAG && H == kDagH && (units == 64 || (units != 16 && N >= kDagWideMinRows))) {
    // ablation bit 2: the input products hoisted into dag_input_gemm_kernel
    out.fn = (knob(CORTEX_KNOB_ABLATE) & 4) ? dag_slice64_kernel<true> : dag_slice64_kernel<false>;
    out.ablate_bits = 4;
    out.J = kDagJ;
    out.threads = kFwdThreads;
    out.lds = kDagListBytes;
    out.level_range_ok = true;
    return true;
  }
#define CORTEX_CASE(CELLID, HH)                                      \
  if (cell == CELLID && H == HH) {                                    \
    pick_slice<CELLID, HH, Cell<CELLID, HH>::J>(cached, out);         \
    return true;                                                      \
  }
  CORTEX_CASE(CORTEX_TREE_RNN, 64)
  CORTEX_CASE(CORTEX_TREE_RNN, 256)
  CORTEX_CASE(CORTEX_NARY_TREELSTM, 64)
  CORTEX_CASE(CORTEX_NARY_TREELSTM, 256)
  CORTEX_CASE(CORTEX_CHILDSUM_TREELSTM, 64)
  CORTEX_CASE(CORTEX_CHILDSUM_TREELSTM, 256)
  CORTEX_CASE(CORTEX_CHILDSUM_TREELSTM, 512)
  CORTEX_CASE(CORTEX_TREE_RNN, 512)
  CORTEX_CASE(CELL_DAG, 64)
  CORTEX_CASE(CELL_DAG, 256)
  CORTEX_CASE(CELL_DAG, 512)
#undef CORTEX_CASE
  if ((cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU) && (H == 64 || H == 256 || H == 512)) {
    const bool simple = cell == CORTEX_SIMPLE_TREEGRU;
    if (H == 64)
      out.fn = simple ? (cached ? treegru_forward_kernel<64, true, true> : treegru_forward_kernel<64, true, false>)
                      : (cached ? treegru_forward_kernel<64, false, true> : treegru_forward_kernel<64, false, false>);
    else if (H == 256)
      out.fn = simple ? (cached ? treegru_forward_kernel<256, true, true> : treegru_forward_kernel<256, true, false>)
                      : (cached ? treegru_forward_kernel<256, false, true> : treegru_forward_kernel<256, false, false>);
    else
      out.fn = simple ? (cached ? treegru_forward_kernel<512, true, true> : treegru_forward_kernel<512, true, false>)
                      : (cached ? treegru_forward_kernel<512, false, true> : treegru_forward_kernel<512, false, false>);
    out.J = 4;
    out.threads = kFwdThreads;
    out.level_barrier_ok = out.level_range_ok = out.phase_barrier_ok = true;
    return true;
  }
  if (cell == CORTEX_MVRNN && H == kMvD) {
    out.fn = mvrnn_forward_kernel<kMvD, false>;
    out.J = MvDims<kMvD>::RB;
    out.threads = MvDims<kMvD>::kThreads;
    out.lds = N <= MvDims<kMvD>::kCacheRows ? 3 * (size_t)N * sizeof(int) : 0;
    return true;
  }
  if (cell == CORTEX_MVRNN && H == kMvD2) {
    out.fn = mvrnn_forward_kernel<kMvD2, false>;
    out.J = MvDims<kMvD2>::RB;
    out.threads = MvDims<kMvD2>::kThreads;
    out.lds = N <= MvDims<kMvD2>::kCacheRows ? 3 * (size_t)N * sizeof(int) : 0;
    return true;
  }
  return false;
}

// The fused instance (linearization inside the forward launch) for a cell
// and hidden size, at the default schedule; false where there is none.
static bool pick_fused(int cell, int H, int32_t N, int32_t K, Instance &out) {
  const int64_t units = knob(CORTEX_KNOB_FWD_SLICE_UNITS);
  if (N > kFusedMaxNodes) return false;
  out.threads = kFwdThreads;
  if (cell == CORTEX_TREE_RNN && H == kLdsH) {
    if (knob(CORTEX_KNOB_TREE_UNROLL) != 0 || N > kLdsMaxRows || knob(CORTEX_KNOB_FWD_NODE_GROUPS) > 1) return false;
    out.fn = tree_rnn_lds_kernel<true>;
    out.J = kLdsH;
    out.one_group = true;
    out.lds = (size_t)N * kLdsHStride * sizeof(float) + fused_struct_ints(N, K) * sizeof(int);
    return true;
  }
  if ((cell == CORTEX_NARY_TREELSTM && (H == 64 || H == 256)) || (cell == CORTEX_TREE_RNN && (H == 256 || H == 512))) {
    const int J = cell == CORTEX_NARY_TREELSTM ? 4 : 16;
    if ((units != 0 && units != J) || K != 2 || N > kMaxCachedRows) return false;
    if (cell == CORTEX_NARY_TREELSTM)
      out.fn = H == 64 ? slice_forward_kernel<CORTEX_NARY_TREELSTM, 64, 4, true, false, true>
                       : slice_forward_kernel<CORTEX_NARY_TREELSTM, 256, 4, true, false, true>;
    else
      out.fn = H == 256 ? slice_forward_kernel<CORTEX_TREE_RNN, 256, 16, true, false, true>
                        : slice_forward_kernel<CORTEX_TREE_RNN, 512, 16, true, false, true>;
    out.J = J;
    out.lds = fused_lds_ints(N, K) * sizeof(int);
    return true;
  }
  if (cell == CELL_DAG && (H == 64 || H == 256 || H == 512)) {
    // the slice kernel with 16-unit slices (at H = 256 the batches below the
    // 64-unit kernel's range)
    if ((units != 0 && units != 16) || K != 2 || N > kMaxCachedRows) return false;
    if (H == 256 && units == 0 && N >= kDagWideMinRows) return false;
    out.fn = H == 64 ? slice_forward_kernel<CELL_DAG, 64, 16, true, false, true>
                     : (H == 256 ? slice_forward_kernel<CELL_DAG, 256, 16, true, false, true>
                                 : slice_forward_kernel<CELL_DAG, 512, 16, true, false, true>);
    out.J = 16;
    out.lds = fused_lds_ints(N, K) * sizeof(int);
    return true;
  }
  if (cell == CORTEX_MVRNN && (H == kMvD || H == kMvD2) && K == 2) {
    out.fn = H == kMvD ? mvrnn_forward_kernel<kMvD, true> : mvrnn_forward_kernel<kMvD2, true>;
    out.J = H == kMvD ? MvDims<kMvD>::RB : MvDims<kMvD2>::RB;
    out.threads = H == kMvD ? MvDims<kMvD>::kThreads : MvDims<kMvD2>::kThreads;
    out.lds = (H == kMvD ? mv_fused_ints<kMvD>(N) : mv_fused_ints<kMvD2>(N)) * sizeof(int);
    return true;
  }
  const bool gru = cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU;
  if ((cell == CORTEX_CHILDSUM_TREELSTM || gru) && (H == 64 || H == 256 || H == 512)) {
    if (units != 0 && units != 4) return false;
    const bool simple = cell == CORTEX_SIMPLE_TREEGRU;
    if (!gru)
      out.fn = H == 64 ? childsum_forward_kernel<64, true, true>
                       : (H == 256 ? childsum_forward_kernel<256, true, true> : childsum_forward_kernel<512, true, true>);
    else if (H == 64)
      out.fn = simple ? treegru_forward_kernel<64, true, true, true> : treegru_forward_kernel<64, false, true, true>;
    else if (H == 256)
      out.fn = simple ? treegru_forward_kernel<256, true, true, true> : treegru_forward_kernel<256, false, true, true>;
    else
      out.fn = simple ? treegru_forward_kernel<512, true, true, true> : treegru_forward_kernel<512, false, true, true>;
    out.J = 4;
    out.lds = fused_struct_ints(N, K) * sizeof(int);
    return true;
  }
  return false;
}

// Workspace of a forward launch: barrier words, the trace area, then the
// tagged staging of h (and of c for the LSTM cells, of P for MV-RNN), 8 bytes
// per element.
static size_t staging_bytes(int32_t N, int32_t H) { return align_up((size_t)N * H * 8, 256); }
static size_t staging_offset() { return align_up(kSyncBytes + kTraceBytes, 256); }
size_t trace_offset() { return kSyncBytes; }
size_t forward_header_bytes() { return staging_offset(); }
static int staged_tensors(int32_t cell) {
  if (cell == CORTEX_NARY_TREELSTM || cell == CORTEX_CHILDSUM_TREELSTM || cell == CORTEX_MVRNN ||
      cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU)
    return 2;                                   // h, and c / P / the TreeGRU reset sum m
  if (cell == CORTEX_TREE_RNN || cell == -1) return 1;
  return 0;
}
// bytes of the second staged tensor: c [N, H], P [N, H, H] for MV-RNN, or the
// TreeGRU reset sums m [N, H] followed by the kept phase-A values [3, N, H]
static size_t keep_bytes(int32_t N, int32_t H) { return align_up((size_t)N * H * 3 * sizeof(float), 256); }
static size_t second_staging_bytes(int32_t cell, int32_t N, int32_t H) {
  if (cell == CORTEX_MVRNN) return align_up((size_t)N * H * H * 8, 256);
  if (cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU) return staging_bytes(N, H) + keep_bytes(N, H);
  return staging_bytes(N, H);
}
// Where a forward launch keeps its header (barrier words, staging epoch,
// entered words; then the trace area in trace builds), its tagged staging of
// h and of the second state (c, P or the TreeGRU reset sums m) and the
// TreeGRU phase values.  The staging regions must only ever have held tagged
// pairs written through this header's epoch, so that every tag in them is at
// most the epoch.
static size_t regions_bytes(int32_t cell, int32_t N, int32_t H, size_t &hs_off, size_t &cs_off, size_t &keep_off) {
  const int staged = staged_tensors(cell == CELL_DAG ? -1 : cell);
  hs_off = staging_offset();
  cs_off = hs_off + (staged >= 1 ? staging_bytes(N, H) : 0);
  keep_off = cs_off + (staged >= 2 ? (cell == CORTEX_MVRNN ? align_up((size_t)N * H * H * 8, 256) : staging_bytes(N, H))
                                   : 0);
  return cortex_forward_workspace_bytes(cell == CELL_DAG ? -1 : cell, N, H);
}

// The regions of a caller's workspace: header, h staging, second staging,
// then the TreeGRU phase values, back to back.
static FwdRegions workspace_regions(void *d_ws, int32_t cell, int32_t N, int32_t H) {
  size_t hs_off, cs_off, keep_off;
  regions_bytes(cell, N, H, hs_off, cs_off, keep_off);
  char *base = (char *)d_ws;
  const int staged = staged_tensors(cell == CELL_DAG ? -1 : cell);
  return FwdRegions{d_ws, staged >= 1 ? base + hs_off : nullptr, staged >= 2 ? base + cs_off : nullptr,
                    (float *)(base + keep_off)};
}

// fused_children != nullptr: the fused instance, which linearizes the batch
// itself and writes *lin; where there is none, or it does not fit one compute
// unit, nothing is enqueued and *launched stays false.  fixed != nullptr: the
// regions come from the caller (ws_bytes is then not checked).
static int launch_forward(int cell, int H, const cortex_lin_t *lin, FwdArgs &a, void *d_ws, size_t ws_bytes,
                          void *stream, const int32_t *fused_children = nullptr, bool *launched = nullptr,
                          const FwdRegions *fixed = nullptr, bool dry_run = false) {
  if (launched) *launched = false;
  // state and staging arrays are addressed with 32-bit byte offsets
  const uint64_t state_bytes = (uint64_t)lin->num_nodes * H * (cell == CORTEX_MVRNN ? H : 1) * 8;
  const uint64_t table_bytes = (uint64_t)(a.x_rows > 0 ? a.x_rows : 0) * H * (cell == CORTEX_MVRNN ? H : 1) * 4;
  if (state_bytes > 0x7fffffffull || table_bytes > 0x7fffffffull) return CORTEX_E_TOO_LARGE;
  if (!fixed && ws_bytes < cortex_forward_workspace_bytes(cell == CELL_DAG ? -1 : cell, lin->num_nodes, H))
    return CORTEX_E_WORKSPACE;
  const FwdRegions reg = fixed ? *fixed : workspace_regions(d_ws, cell, lin->num_nodes, H);
  size_t dyn = 0;
  bool cached = false;
  Instance inst;
  if (fused_children) {
    if (knob(CORTEX_KNOB_LIN_BLOCKS) != 0 || knob(CORTEX_KNOB_LEVEL_SYNC) != 0 || knob(CORTEX_KNOB_ABLATE) != 0 ||
        !pick_fused(cell, H, lin->num_nodes, lin->max_arity, inst))
      return CORTEX_OK;
    dyn = inst.lds;
  } else if (cell != CORTEX_MVRNN) {
    dyn = cache_ints(cell, lin->num_nodes, lin->max_arity) * sizeof(int);
    const bool childsum_like =
        cell == CORTEX_CHILDSUM_TREELSTM || cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU;
    cached = dyn <= kStructCacheBudget && (childsum_like || lin->num_nodes <= kMaxCachedRows);
    if (!cached) dyn = 0;
  }
  if (!fused_children) {
    if (!pick(cell, H, lin->num_nodes, cached, inst)) return CORTEX_E_INVAL;
    if (inst.lds != SIZE_MAX) dyn = inst.lds;
  }
  const int per_cu = cached_occupancy((const void *)inst.fn, inst.threads, dyn);
  const int cus = num_cus();
  if (cus <= 0) return CORTEX_E_HIP;
  if (per_cu <= 0) return fused_children ? CORTEX_OK : CORTEX_E_HIP;
  const int cap = per_cu * cus;
  int S;
  int64_t q = knob(CORTEX_KNOB_FWD_NODE_GROUPS);
  if (cell == CORTEX_MVRNN) {
    S = inst.J;                       // row blocks of P per node
    if (q <= 0) q = cus / S;
  } else {
    // one slice (TreeRNN at H = 64) or one workgroup per tree: a node group
    // per 16 nodes, up to one per compute unit; else fill the GPU with slices
    S = H / inst.J;
    if (q <= 0) q = S == 1 ? std::min<int64_t>(cus, ((int64_t)lin->num_nodes + 15) / 16) : cus / S;
    if (inst.one_group) q = 1;
  }
  if (q < 1) q = 1;
  const int64_t G = S * q;
  if (G > cap || G > kMaxGrid) return CORTEX_E_TOO_LARGE;
  a.S = S;
  a.Q = (int32_t)q;
  a.sync = (unsigned int *)reg.header;
  a.trace = (uint64_t *)((char *)reg.header + kSyncBytes);
  a.timeout = barrier_timeout_ticks();
  a.hs = reg.hs;
  a.cs = reg.cs;                                     // c, P for MV-RNN, or the TreeGRU reset sums
  a.keep = inst.phase_barrier_ok ? reg.keep : nullptr;
  a.retire = 1;                 // the tag itself comes from the workspace header (launch_tag)
  a.level_lo = 0;
  a.level_hi = 0x7fffffff;
  a.level_barrier = 0;
  const int64_t sync_mode = knob(CORTEX_KNOB_LEVEL_SYNC);
  if ((sync_mode == 1 && !inst.level_barrier_ok) || (sync_mode == 2 && !inst.level_range_ok) ||
      (sync_mode == 3 && !inst.phase_barrier_ok))
    return CORTEX_E_INVAL;
  const int64_t ablate = knob(CORTEX_KNOB_ABLATE);
  if (ablate & ~(int64_t)inst.ablate_bits) return CORTEX_E_INVAL;
  if (dry_run) {                      // every host check passed; enqueue nothing
    if (fused_children) *launched = true;
    return CORTEX_OK;
  }
  a.ablate = (int32_t)ablate;
  set_last_grid(1, (int32_t)G);
  if (ablate & 4) {
    // hoisted input products: W x + b of every row goes to the output rows
    // first; the level loop reads each element there just before it writes
    // the element's state (the same thread, so no other ordering is needed)
    a.pre = a.h;
    const int blocks = (int)(((int64_t)lin->num_nodes + kFwdWaves * kTileM - 1) / (kFwdWaves * kTileM));
    const int grid = (blocks * kDagS + 31) / 32 * 32;
    void *kargs[] = {(void *)&a};
    if (grid > 0 && hipLaunchKernel((const void *)dag_input_gemm_kernel, dim3(grid), dim3(kFwdThreads), kargs, 0,
                                    (hipStream_t)stream) != hipSuccess)
      return CORTEX_E_HIP;
  }
  if (sync_mode == 1) a.level_barrier = 1;
  if (sync_mode == 3) a.level_barrier = 2;
  if (fused_children) {
    a.children = fused_children;
    a.o_num_levels = lin->num_levels;
    a.o_height = lin->height;
    a.o_level_offsets = lin->level_offsets;
    a.o_level_nodes = lin->level_nodes;
    a.o_node_row = lin->node_row;
    a.o_child_rows = lin->child_rows;
    set_last_grid(0, 0);
    *launched = true;
  }
  if (sync_mode != 2) return launch_persistent(inst.fn, (int)G, inst.threads, dyn, a, stream);
  // one launch per level (ablation): L is read back first; every launch
  // reloads weights and structure and reads the same staging epoch (only the
  // last one advances it), so all use one tag and a level reads what the
  // previous launches staged
  int32_t L = 0;
  if (hipMemcpyAsync(&L, lin->num_levels, sizeof(L), hipMemcpyDeviceToHost, (hipStream_t)stream) != hipSuccess ||
      hipStreamSynchronize((hipStream_t)stream) != hipSuccess)
    return CORTEX_E_HIP;
  if (L < 1 || L > lin->num_nodes) L = 1;          // the kernel itself reports a broken linearization
  for (int32_t l = 0; l < L; ++l) {
    a.level_lo = l;
    a.level_hi = l + 1;
    a.retire = l == L - 1;
    const int rc = launch_persistent(inst.fn, (int)G, inst.threads, dyn, a, stream);
    if (rc != CORTEX_OK) return rc;
  }
  return CORTEX_OK;
}

static void fill_lin(FwdArgs &a, const cortex_lin_t *lin) {
  a.N = lin->num_nodes;
  a.K = lin->max_arity;
  a.num_levels = lin->num_levels;
  a.level_offsets = lin->level_offsets;
  a.level_nodes = lin->level_nodes;
  a.child_rows = lin->child_rows;
}

static bool lin_ok(const cortex_lin_t *lin) {
  return lin && lin->num_nodes >= 0 && lin->max_arity >= 1 && lin->max_arity <= 4 && lin->num_levels &&
         lin->level_offsets && lin->level_nodes && lin->child_rows;
}

}  // namespace cortex

using namespace cortex;


extern "C" size_t cortex_forward_workspace_bytes(int32_t cell, int32_t N, int32_t H) {
  if (N < 0 || H <= 0) return 0;
  if (cell < -1 || cell > CORTEX_SIMPLE_TREEGRU) return 0;
  const int staged = cortex::staged_tensors(cell);
  return cortex::staging_offset() + (staged >= 1 ? cortex::staging_bytes(N, H) : 0) +
         (staged >= 2 ? cortex::second_staging_bytes(cell, N, H) : 0);
}

// Host checks of a tree forward's arguments (N > 0) and its argument block.
static int tree_args(int32_t cell, const cortex_lin_t *lin, const float *d_x_table, int32_t x_rows,
                     const int32_t *d_x_index, const float *d_leaf_mat, const cortex_weights_t *w, float *d_h,
                     float *d_c_or_P, int32_t *d_status, void *d_ws, FwdArgs &a) {
  if (!d_ws || !d_h || !d_x_index || (x_rows > 0 && !d_x_table)) return CORTEX_E_INVAL;
  const int K = lin->max_arity;
  if (cell == CORTEX_CHILDSUM_TREELSTM) {
    if (!w->W || !w->U || !w->b || !d_c_or_P) return CORTEX_E_INVAL;
  } else if (cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU) {
    if (!w->W || !w->U || !w->b) return CORTEX_E_INVAL;
  } else {
    if (K != 2) return CORTEX_E_INVAL;
    if (cell == CORTEX_TREE_RNN && (!w->W || !w->b)) return CORTEX_E_INVAL;
    if (cell == CORTEX_NARY_TREELSTM && (!w->U || !w->b || !d_c_or_P)) return CORTEX_E_INVAL;
    if (cell == CORTEX_MVRNN && (!w->W || !w->W_M || !d_c_or_P || (x_rows > 0 && !d_leaf_mat)))
      return CORTEX_E_INVAL;
  }
  a = FwdArgs{};
  fill_lin(a, lin);
  a.x_rows = x_rows;
  a.x_table = d_x_table;
  a.x_index = d_x_index;
  a.leaf_mat = d_leaf_mat;
  a.W = w->W;
  a.U = w->U;
  a.b = w->b;
  a.W_M = w->W_M;
  a.h = d_h;
  a.c = d_c_or_P;
  a.status = d_status;
  return CORTEX_OK;
}

namespace cortex {

static int tree_forward_impl(int32_t cell, int32_t H, const cortex_lin_t *lin, const float *d_x_table,
                             int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                             const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status, void *d_ws,
                             size_t ws_bytes, void *stream, const FwdRegions *fixed, bool dry_run) {
  if (!lin_ok(lin) || !w || !d_status || x_rows < 0) return CORTEX_E_INVAL;
  if (cell < CORTEX_TREE_RNN || cell > CORTEX_SIMPLE_TREEGRU) return CORTEX_E_INVAL;
  if (lin->num_nodes == 0) return CORTEX_OK;
  FwdArgs a;
  const int rc = tree_args(cell, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P, d_status, d_ws, a);
  if (rc != CORTEX_OK) return rc;
  return launch_forward(cell, H, lin, a, d_ws, ws_bytes, stream, nullptr, nullptr, fixed, dry_run);
}

// The whole path of a tree batch: one fused launch where there is an
// instance for it, else the linearizer then the forward.  lin_ws / fwd_ws are
// the two workspaces (fixed: the forward's regions, placed by the caller).
// dry_run: every host check, nothing enqueued.
int tree_infer_impl(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                    const float *d_x_table, int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                    const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status, void *lin_ws,
                    size_t lin_ws_bytes, void *fwd_ws, size_t fwd_ws_bytes, const FwdRegions *fixed, void *stream,
                    bool dry_run) {
  const int32_t N = lin->num_nodes, K = lin->max_arity;
  if (N == 0) return linearize_impl(d_children, 0, K, lin, d_status, lin_ws, lin_ws_bytes, stream, dry_run);
  if (!d_children) return CORTEX_E_INVAL;
  FwdArgs a;
  int rc = tree_args(cell, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P, d_status, fwd_ws, a);
  if (rc != CORTEX_OK) return rc;
  // one launch where a fused instance exists and fits; else the two calls
  bool launched = false;
  rc = launch_forward(cell, H, lin, a, fwd_ws, fwd_ws_bytes, stream, d_children, &launched, fixed, dry_run);
  if (rc != CORTEX_OK || launched) return rc;
  rc = linearize_impl(d_children, N, K, lin, d_status, lin_ws, lin_ws_bytes, stream, dry_run);
  if (rc != CORTEX_OK) return rc;
  return tree_forward_impl(cell, H, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P, d_status,
                           fwd_ws, fwd_ws_bytes, stream, fixed, dry_run);
}

// Regions of the forward for a workspace placed by the library (the
// allocation-free entry point): the header and each staging region at their
// own fixed offsets, whatever the batch, so a region only ever holds its own
// kind of data.
bool fixed_regions(int32_t cell, int32_t N, int32_t H, void *header, size_t header_cap, void *hs, size_t hs_cap,
                   void *cs, size_t cs_cap, void *keep, size_t keep_cap, FwdRegions &out) {
  size_t hs_off, cs_off, keep_off;
  regions_bytes(cell, N, H, hs_off, cs_off, keep_off);
  const int staged = staged_tensors(cell);
  const size_t need_hs = staged >= 1 ? cs_off - hs_off : 0;
  const size_t need_cs = staged >= 2 ? keep_off - cs_off : 0;
  const size_t need_keep = (cell == CORTEX_CHILDSUM_TREEGRU || cell == CORTEX_SIMPLE_TREEGRU) ? keep_bytes(N, H) : 0;
  if (hs_off > header_cap || need_hs > hs_cap || need_cs > cs_cap || need_keep > keep_cap) return false;
  out = FwdRegions{header, staged >= 1 ? hs : nullptr, staged >= 2 ? cs : nullptr, (float *)keep};
  return true;
}

}  // namespace cortex

extern "C" int cortex_tree_forward(int32_t cell, int32_t H, const cortex_lin_t *lin, const float *d_x_table,
                                   int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                                   const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status,
                                   void *d_ws, size_t ws_bytes, void *stream) {
  return tree_forward_impl(cell, H, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P, d_status, d_ws,
                           ws_bytes, stream, nullptr, false);
}

extern "C" int cortex_dag_forward(int32_t H, const cortex_lin_t *lin, const float *d_x, const float *d_W,
                                  const float *d_U, const float *d_b, float *d_h, int32_t *d_status, void *d_ws,
                                  size_t ws_bytes, void *stream) {
  if (!lin_ok(lin) || !d_status) return CORTEX_E_INVAL;
  if (lin->max_arity != 2) return CORTEX_E_INVAL;
  if (lin->num_nodes == 0) return CORTEX_OK;
  if (!d_x || !d_W || !d_U || !d_b || !d_h || !d_ws) return CORTEX_E_INVAL;
  FwdArgs a = {};
  fill_lin(a, lin);
  a.x = d_x;
  a.W = d_W;
  a.U = d_U;
  a.b = d_b;
  a.h = d_h;
  a.status = d_status;
  return launch_forward(CELL_DAG, H, lin, a, d_ws, ws_bytes, stream);
}

extern "C" size_t cortex_tree_infer_workspace_bytes(int32_t cell, int32_t N, int32_t K, int32_t H) {
  if (cell < CORTEX_TREE_RNN || cell > CORTEX_SIMPLE_TREEGRU) return 0;
  const size_t lw = cortex_linearize_workspace_bytes(N, K), fw = cortex_forward_workspace_bytes(cell, N, H);
  if (lw == 0 || fw == 0) return 0;
  return align_up(lw, 256) + fw;
}

extern "C" int cortex_tree_infer(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                                 const float *d_x_table, int32_t x_rows, const int32_t *d_x_index,
                                 const float *d_leaf_mat, const cortex_weights_t *w, float *d_h, float *d_c_or_P,
                                 int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream) {
  if (!lin_ok(lin) || !w || !d_status || x_rows < 0 || !lin->height || !lin->node_row) return CORTEX_E_INVAL;
  if (cell < CORTEX_TREE_RNN || cell > CORTEX_SIMPLE_TREEGRU) return CORTEX_E_INVAL;
  const int32_t N = lin->num_nodes, K = lin->max_arity;
  if (N == 0) return cortex_linearize(d_children, 0, K, lin, d_status, d_ws, ws_bytes, stream);
  if (!d_children) return CORTEX_E_INVAL;
  FwdArgs a;
  const int rc = tree_args(cell, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P, d_status, d_ws, a);
  if (rc != CORTEX_OK) return rc;
  const size_t need = cortex_tree_infer_workspace_bytes(cell, N, K, H);
  if (need == 0) return CORTEX_E_INVAL;
  if (ws_bytes < need) return CORTEX_E_WORKSPACE;
  const size_t lw = align_up(cortex_linearize_workspace_bytes(N, K), 256);
  return tree_infer_impl(cell, H, d_children, lin, d_x_table, x_rows, d_x_index, d_leaf_mat, w, d_h, d_c_or_P,
                         d_status, d_ws, lw, (char *)d_ws + lw, ws_bytes - lw, nullptr, stream, false);
}

extern "C" size_t cortex_dag_infer_workspace_bytes(int32_t N, int32_t K, int32_t H) {
  const size_t lw = cortex_linearize_workspace_bytes(N, K), fw = cortex_forward_workspace_bytes(-1, N, H);
  if (lw == 0 || fw == 0) return 0;
  return align_up(lw, 256) + fw;
}

extern "C" int cortex_dag_infer(int32_t H, const int32_t *d_children, const cortex_lin_t *lin, const float *d_x,
                                const float *d_W, const float *d_U, const float *d_b, float *d_h,
                                int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream) {
  if (!lin_ok(lin) || !d_status || !lin->height || !lin->node_row) return CORTEX_E_INVAL;
  if (lin->max_arity != 2) return CORTEX_E_INVAL;
  const int32_t N = lin->num_nodes, K = lin->max_arity;
  if (N == 0) return cortex_linearize(d_children, 0, K, lin, d_status, d_ws, ws_bytes, stream);
  if (!d_children || !d_x || !d_W || !d_U || !d_b || !d_h || !d_ws) return CORTEX_E_INVAL;
  const size_t need = cortex_dag_infer_workspace_bytes(N, K, H);
  if (need == 0) return CORTEX_E_INVAL;
  if (ws_bytes < need) return CORTEX_E_WORKSPACE;
  const size_t lw = align_up(cortex_linearize_workspace_bytes(N, K), 256);
  void *fws = (char *)d_ws + lw;
  const size_t fws_bytes = ws_bytes - lw;
  FwdArgs a = {};
  fill_lin(a, lin);
  a.x = d_x;
  a.W = d_W;
  a.U = d_U;
  a.b = d_b;
  a.h = d_h;
  a.status = d_status;
  bool launched = false;
  int rc = launch_forward(CELL_DAG, H, lin, a, fws, fws_bytes, stream, d_children, &launched);
  if (rc != CORTEX_OK || launched) return rc;
  rc = cortex_linearize(d_children, N, K, lin, d_status, d_ws, lw, stream);
  if (rc != CORTEX_OK) return rc;
  return cortex_dag_forward(H, lin, d_x, d_W, d_U, d_b, d_h, d_status, fws, fws_bytes, stream);
}
