// Persistent level-synchronous forward kernels (Sec. 4.1 loop nest; kernel
// fusion and model persistence as evaluated in Sec. 7.2-7.3).
//
// One launch runs every level.  Workgroup b owns hidden slice s = b % S
// (J hidden units, all gates of those units) and node group q = b / S.  Its
// slice of the cell weights is loaded into LDS once and stays there for the
// whole pass (persistence).  Rows are cut into 16-row tiles on a fixed grid
// (tile t = rows [16t, 16t+16)); at level l, group q takes the tiles t = q
// (mod Q) that intersect the level's rows.  For a tile, each of the 8 waves
// loads its share of the input rows (child states, and the node input where
// the cell fuses it) straight into registers in the MFMA operand layout,
// contracts it with the resident weight slice on the fp32 MFMA units, and the
// partial sums meet in LDS for the gate nonlinearities, which write the
// slice's J columns of the new states.  The next tile's rows are requested
// before the current tile's contraction, so load latency overlaps compute.
//
// A device-wide barrier separates levels (the dependence is carried by the
// level loop only, Appendix A.4).  States written by other workgroups move
// through device-scope loads and stores (DevBuf), so the barrier needs no L2
// write-back or invalidate.  TreeRNN and N-ary TreeLSTM leaves are the inputs
// themselves (specialization, Sec. 3.1; zero initial memory cell, Sec. 4.3):
// a level reading a leaf child takes the row from the input table directly,
// which removes the barrier after the leaf level.
#include <atomic>

#include "cortex_device.hpp"
#include "cortex_host.hpp"

namespace cortex {

constexpr int kFwdThreads = 512;
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kTileM = 16;
constexpr int CELL_DAG = 16;                 // internal id of the DAG-RNN cell

// Optional timeline (builds with -DCORTEX_TRACE only): every workgroup (up to
// kTraceBlocks) stamps the 100 MHz wall clock at phase boundaries of every
// level into trace[block][kTraceLevels][8] (uint64), placed in the workspace
// after the barrier words.  Row kTraceLevels-1 holds kernel-wide stamps:
// entry, weights loaded, structure ready, exit.
constexpr int kTraceLevels = 64;
constexpr int kTraceBlocks = 256;
#ifdef CORTEX_TRACE
constexpr size_t kTraceBytes = (size_t)kTraceBlocks * kTraceLevels * 8 * sizeof(uint64_t);
#define CORTEX_TRACE_AT(row, k)                                                              \
  do {                                                                                      \
    if (threadIdx.x == 0 && blockIdx.x < kTraceBlocks)                                      \
      a.trace[((size_t)blockIdx.x * kTraceLevels + (row)) * 8 + (k)] = wall_clock64();       \
  } while (0)
#define CORTEX_TRACE_POINT(lvl, k) CORTEX_TRACE_AT(min((lvl), kTraceLevels - 2), k)
#define CORTEX_TRACE_KERNEL(k) CORTEX_TRACE_AT(kTraceLevels - 1, k)
#else
constexpr size_t kTraceBytes = 0;
#define CORTEX_TRACE_POINT(lvl, k) \
  do {                             \
  } while (0)
#define CORTEX_TRACE_KERNEL(k) \
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
  uint32_t tag;                 // this launch's staging tag
  void *hs, *cs;                // tagged staging of h and c (workspace)
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

template <int CELL, int H>
struct Cfg;
template <int H>
struct Cfg<CORTEX_TREE_RNN, H> {
  static constexpr int J = (H <= 64) ? H : 16, GATES = 1, KA = 2 * H;
};
template <int H>
struct Cfg<CORTEX_NARY_TREELSTM, H> {
  static constexpr int J = 4, GATES = 5, KA = 2 * H;
};
template <int H>
struct Cfg<CORTEX_CHILDSUM_TREELSTM, H> {
  static constexpr int J = 4, GATES = 4, KA = 2 * H;
};
template <int H>
struct Cfg<CELL_DAG, H> {
  static constexpr int J = 16, GATES = 1, KA = 3 * H;
};

template <int CELL, int H>
struct Dims {
  using C = Cfg<CELL, H>;
  static constexpr int J = C::J, GATES = C::GATES, KA = C::KA;
  static constexpr int MPAD = (GATES * J + 15) / 16 * 16;
  static constexpr int NT = MPAD / 16;
  static constexpr bool kChildSum = CELL == CORTEX_CHILDSUM_TREELSTM;
  static constexpr bool kLeafInputs = CELL == CORTEX_TREE_RNN || CELL == CORTEX_NARY_TREELSTM;
  static constexpr bool kCells = CELL == CORTEX_NARY_TREELSTM || CELL == CORTEX_CHILDSUM_TREELSTM;
  // generic path: k range per wave, padded to whole 16-blocks (zeros beyond KA)
  static constexpr int KW = ((KA + kFwdWaves * 16 - 1) / (kFwdWaves * 16)) * 16;
  static constexpr int NB = KW / 16;                       // float4 loads per lane per tile
  // child-sum: node part over 4 waves, edge part (64 edge rows) over 8 waves
  static constexpr int KWX = H / 4, NBX = KWX / 16;
  static constexpr int KWE = H / 2, NBE = KWE / 16;
  static constexpr int LDW = kChildSum ? (2 * H + 4) : (kFwdWaves * KW + 4);   // weight row stride
  static constexpr int C_FLOATS = kChildSum ? (4 * 16 * 16 + 2 * 64 * 16) : kFwdWaves * 16 * MPAD;
  static constexpr int EPI = kTileM * J;                   // epilogue (row, unit) pairs
  static constexpr int EPI_PER_THREAD = (EPI + kFwdThreads - 1) / kFwdThreads;
  static_assert(H % J == 0, "slices must tile H");
  static_assert(H % 64 == 0, "H must be a multiple of 64");
};

// Weight-slice row m = (gate g, unit j); child-sum rows are ordered
// (i, o, u, f) while the input layout is (i, f, o, u).
__device__ __forceinline__ int childsum_gate(int gslot) {
  return gslot == 0 ? 0 : (gslot == 1 ? 2 : (gslot == 2 ? 3 : 1));
}

template <int CELL, int H>
__device__ void load_weight_slice(const FwdArgs &a, int hbase, float *W_s, float *bias_s) {
  using D = Dims<CELL, H>;
  constexpr int ROW4 = (D::LDW - 4) / 4, SEG4 = H / 4, KA4 = D::KA / 4;
  for (int idx = threadIdx.x; idx < D::MPAD * ROW4; idx += kFwdThreads) {
    const int m = idx / ROW4, c4 = idx % ROW4;
    const int g = m / D::J, j = m % D::J, hj = hbase + j;
    const int sg = c4 / SEG4, o4 = c4 % SEG4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (m < D::GATES * D::J && c4 < KA4) {
      const float *src = nullptr;
      if (CELL == CORTEX_TREE_RNN) src = a.W + (size_t)hj * 2 * H + sg * H;
      if (CELL == CORTEX_NARY_TREELSTM) src = a.U + ((size_t)(sg * 5 + g) * H + hj) * H;
      if (CELL == CORTEX_CHILDSUM_TREELSTM)
        src = (sg == 0 ? a.W : a.U) + ((size_t)childsum_gate(g) * H + hj) * H;
      if (CELL == CELL_DAG) src = (sg == 0 ? a.W : a.U + (size_t)(sg - 1) * H * H) + (size_t)hj * H;
      v = *(const float4 *)(src + o4 * 4);
    }
    *(float4 *)&W_s[m * D::LDW + c4 * 4] = v;
  }
  for (int m = threadIdx.x; m < D::MPAD; m += kFwdThreads) {
    const int g = m / D::J, j = m % D::J, hj = hbase + j;
    float v = 0.f;
    if (m < D::GATES * D::J) {
      if (CELL == CORTEX_TREE_RNN || CELL == CELL_DAG) v = a.b[hj];
      if (CELL == CORTEX_NARY_TREELSTM) v = a.b[g * H + hj];
      if (CELL == CORTEX_CHILDSUM_TREELSTM) v = a.b[childsum_gate(g) * H + hj];
    }
    bias_s[m] = v;
  }
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
  for (int l = threadIdx.x; kCached && l < L; l += kFwdThreads) {
    const int o0 = st.offset(l), o1 = st.offset(l + 1);
    if (o1 < o0 || (l == 0 && o0 != 0) || (l == L - 1 && o1 != N)) bad = 1;
  }
  // every child row lies in a strictly lower level than its parent row; the
  // level of a row is found by binary search over the offsets.  (Uncached
  // structures are checked tile by tile as the level loop reads them.)
  for (int r = threadIdx.x; kCached && r < N && !bad; r += kFwdThreads) {
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

// Input row of row r (cached, or through level_nodes and x_index).
template <bool kCached>
__device__ __forceinline__ int input_row_of(const FwdArgs &a, const Structure<kCached> &st, int r) {
  if (kCached) return st.input_row(r);
  const int v = a.level_nodes[r];
  if (v < 0 || v >= a.N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return -1;
  }
  const int xi = a.x_index[v];
  if (xi < -1 || xi >= a.x_rows) {
    raise_status(a.status, CORTEX_ST_INPUT_RANGE);
    return -1;
  }
  return xi;
}

// Structure of up to kChunkTiles of a workgroup's tiles in one level, staged
// into LDS in one round trip when the whole linearization is not cached: the
// operand addresses of a tile then never wait on a global load.
constexpr int kChunkTiles = 16;
struct ChunkRows {
  int crow[kChunkTiles][kTileM][4];
  int node[kChunkTiles][kTileM];
  int xrow[kChunkTiles][kTileM];
};

template <bool kNeedX, bool kNeedNode>
__device__ void stage_chunk(const FwdArgs &a, ChunkRows &cr, int c0, int ntiles, int Q, int r0, int r1) {
  for (int idx = threadIdx.x; idx < ntiles * kTileM; idx += kFwdThreads) {
    const int u = idx / kTileM, i = idx % kTileM;
    const int row = (c0 + u * Q) * kTileM + i;
    const bool live = row >= r0 && row < r1;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      int c = (live && s < a.K) ? a.child_rows[(size_t)row * a.K + s] : -1;
      if (c < -1 || c >= r0) {                    // a child must sit in a lower level
        raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
        c = -1;
      }
      cr.crow[u][i][s] = c;
    }
    int v = live ? a.level_nodes[row] : -1;
    if (v < -1 || v >= a.N) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      v = -1;
    }
    if (kNeedNode) cr.node[u][i] = v;
    if (kNeedX) {
      int xi = v >= 0 ? a.x_index[v] : -1;
      if (xi < -1 || xi >= a.x_rows) {
        raise_status(a.status, CORTEX_ST_INPUT_RANGE);
        xi = -1;
      }
      cr.xrow[u][i] = xi;
    }
  }
}

// Leaf level of TreeRNN / N-ary TreeLSTM, spread evenly over every thread of
// the launch: h = input row (or 0), c = 0, staged for the level above and
// written to the outputs.
template <int H, bool kCached, bool kWithC>
__device__ void stage_leaves(const FwdArgs &a, const Structure<kCached> &st, const TagBuf &hs, const TagBuf &cs,
                             int r1, uint32_t tag) {
  const int total = r1 * H;
  for (int e = blockIdx.x * kFwdThreads + threadIdx.x; e < total; e += gridDim.x * kFwdThreads) {
    const int r = e / H, col = e % H;
    const int xr = input_row_of(a, st, r);
    const float v = xr >= 0 ? a.x_table[(size_t)xr * H + col] : 0.f;
    hs.store1((uint32_t)e, v, tag);
    a.h[e] = v;
    if (kWithC) {
      cs.store1((uint32_t)e, 0.f, tag);
      a.c[e] = 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// TreeRNN, N-ary TreeLSTM and DAG-RNN.
//   A row of a tile = [h(slot 0) | h(slot 1)]   (TreeRNN, N-ary TreeLSTM)
//                   = [x | h(slot 0) | h(slot 1)]   (DAG-RNN)
// Wave w owns the columns [w*KW, (w+1)*KW) of A (zero beyond KA).
//
// No device-wide barrier: a workgroup moves on to the next level as soon as
// its own tiles are done.  Child states come from the tagged staging buffers
// (hs, cs); a fragment whose tag is not yet this launch's is loaded again
// until it is, with a wall-clock limit.  Levels only read lower levels and
// every workgroup walks the levels upwards, so the waits always end.
// ---------------------------------------------------------------------------
template <int CELL, int H, bool kCached>
__global__ void __launch_bounds__(kFwdThreads) slice_forward_kernel(FwdArgs a) {
  using D = Dims<CELL, H>;
  constexpr int J = D::J, MPAD = D::MPAD, NT = D::NT, LDW = D::LDW, KW = D::KW, NB = D::NB;
  constexpr int KA = D::KA, EPT = D::EPI_PER_THREAD;
  constexpr bool kLeafInputs = D::kLeafInputs;

  __shared__ __attribute__((aligned(16))) float W_s[MPAD * LDW];
  __shared__ __attribute__((aligned(16))) float C_s[D::C_FLOATS];
  __shared__ float bias_s[MPAD];
  __shared__ ChunkRows chunk;
  extern __shared__ int cache[];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int slice = blockIdx.x % a.S, group = blockIdx.x / a.S, Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N;
  const uint32_t tag = a.tag;
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const TagBuf cs(a.cs, a.cs ? (uint32_t)N * H * 8 : 0u);
  const InBuf xin(a.x, a.x ? (uint32_t)N * H * 4 : 0u);

  CORTEX_TRACE_KERNEL(0);
  if (load_status(a.status) != 0) return;
  load_weight_slice<CELL, H>(a, hbase, W_s, bias_s);
  CORTEX_TRACE_KERNEL(1);
  Structure<kCached> st;
  int L;
  if (!setup_structure<kCached, kLeafInputs, CELL == CELL_DAG>(a, cache, st, L)) return;
  CORTEX_TRACE_KERNEL(2);

  for (int l = 0; l < L; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = st.offset(l), r1 = st.offset(l + 1);
    if (!kCached && (r1 < r0 || r1 > N || (l == 0 && r0 != 0))) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int t_lo = r0 / kTileM, t_hi = (r1 - 1) / kTileM;
    const int t_first = t_lo + ((group - t_lo % Q) % Q + Q) % Q;

    if (kLeafInputs && l == 0) {
      stage_leaves<H, kCached, CELL == CORTEX_NARY_TREELSTM>(a, st, hs, cs, r1, tag);
      continue;
    }

    // structure accessors of the current chunk of tiles
    int c0 = t_first;
    auto crow = [&](int t, int i, int s) -> int {
      if (kCached) return s < a.K ? st.child(t * kTileM + i, s) : -1;
      return chunk.crow[(t - c0) / Q][i][s];
    };
    auto node_of = [&](int t, int i) -> int {
      if (kCached) return st.node_of(t * kTileM + i);
      return chunk.node[(t - c0) / Q][i];
    };

    // A fragment of (tile t, lane row i16, wave-uniform k block kk).  Both
    // loads are always issued (an absent source reads zeros); returns the
    // staged element index to wait on, or -1 (raw = plain input or zeros).
    auto load_a = [&](int t, int kk, Frag4 &f, bool &raw) -> int {
      const int row = t * kTileM + i16;
      const bool live = row >= r0 && row < r1 && kk < KA;
      const int sg = kk / H, o = kk % H + 4 * g4;
      const bool is_x = CELL == CELL_DAG && sg == 0;
      uint32_t xoff = kNoSource, soff = kNoSource;
      int e = -1;
      if (live && is_x) {
        const int nd = node_of(t, i16);
        if (nd >= 0 && nd < N) xoff = (uint32_t)((nd * H + o) * 4);
      } else if (live) {
        const int cr = crow(t, i16, CELL == CELL_DAG ? sg - 1 : sg);
        if (cr >= 0) e = cr * H + o;
      }
      if (e >= 0) soff = (uint32_t)e * 8u;
      if (CELL == CELL_DAG) {
        // x blocks and state blocks are wave-uniform; one of the two loads reads zeros
        const u32x4 xv = xin.load4(xoff);
        f.lo = hs.load2_at(soff);
        f.hi = hs.load2_at(soff + 16u);
        if (is_x) f.lo = xv;
      } else {
        f.lo = hs.load2_at(soff);
        f.hi = hs.load2_at(soff + 16u);
      }
      raw = e < 0;
      return e;
    };
    // staged memory cells of the children of epilogue pair e (N-ary only)
    auto load_cc = [&](int t, u32x2 (&cc)[EPT][2], int (&ce)[EPT][2]) {
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          cc[e][s] = u32x2{0u, tag};
          ce[e][s] = -1;
        }
        if (!D::kCells) continue;
        const int p = tid + e * kFwdThreads;
        const int row = t * kTileM + p / J, hj = hbase + p % J;
        const bool live = p < D::EPI && row >= r0 && row < r1;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int cr = live ? crow(t, p / J, s) : -1;
          if (cr >= 0 && cr < r0) ce[e][s] = cr * H + hj;
          cc[e][s] = cs.load1_at(ce[e][s] >= 0 ? (uint32_t)ce[e][s] * 8u : kNoSource);
        }
      }
    };

    Frag4 fa[NB], fn[NB];
    int ea[NB], en[NB];
    bool ra[NB], rn[NB];
    u32x2 cc[EPT][2], ccn[EPT][2];
    int cea[EPT][2], cen[EPT][2];
    for (; c0 <= t_hi; c0 += Q * kChunkTiles) {
    const int c_last = min(t_hi, c0 + Q * (kChunkTiles - 1));
    if (!kCached) {
      __syncthreads();                // the previous chunk's structure is no longer read
      stage_chunk<false, CELL == CELL_DAG>(a, chunk, c0, (c_last - c0) / Q + 1, Q, r0, r1);
      __syncthreads();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) ea[b] = load_a(c0, wave * KW + 16 * b, fa[b], ra[b]);
    load_cc(c0, cc, cea);
    for (int t = c0; t <= c_last; t += Q) {
      const int tn = t + Q;
      if (tn <= c_last) {               // request the next tile before computing this one
#pragma unroll
        for (int b = 0; b < NB; ++b) en[b] = load_a(tn, wave * KW + 16 * b, fn[b], rn[b]);
        load_cc(tn, ccn, cen);
      }
      CORTEX_TRACE_POINT(l, 1);
      // ---- wait for staged fragments that are not this launch's yet: poll
      //      one element, then load the fragment again ----
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (ea[b] >= 0 && !fa[b].staged_ready(tag)) {
          const uint64_t t0 = wall_clock64();
          int naps = 0;
          do {
            while (hs.load1((uint32_t)ea[b] + 3).y != tag && keep_waiting(a.status, t0, a.timeout, naps)) {
            }
            fa[b].lo = hs.load2((uint32_t)ea[b]);
            fa[b].hi = hs.load2((uint32_t)ea[b] + 2);
          } while (!fa[b].staged_ready(tag) && keep_waiting(a.status, t0, a.timeout, naps));
        }
      }
#pragma unroll
      for (int e = 0; e < EPT; ++e)
#pragma unroll
        for (int s = 0; s < 2; ++s)
          if (cea[e][s] >= 0 && cc[e][s].y != tag) {
            const uint64_t t0 = wall_clock64();
            int naps = 0;
            do {
              cc[e][s] = cs.load1((uint32_t)cea[e][s]);
            } while (cc[e][s].y != tag && keep_waiting(a.status, t0, a.timeout, naps));
          }
      CORTEX_TRACE_POINT(l, 2);
      // ---- contraction: partial sums of this wave's k range ----
      floatx4 acc0[NT], acc1[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc0[nt] = acc1[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
      const float *brow = &W_s[i16 * LDW + wave * KW + 4 * g4];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float4 av = fa[b].value(ra[b]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const float4 bv = *(const float4 *)(brow + nt * 16 * LDW + 16 * b);
          if (b & 1) acc1[nt] = mfma_k16(av, bv, acc1[nt]);
          else acc0[nt] = mfma_k16(av, bv, acc0[nt]);
        }
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          C_s[(wave * 16 + 4 * g4 + v) * MPAD + nt * 16 + i16] = acc0[nt][v] + acc1[nt][v];
      __syncthreads();
      CORTEX_TRACE_POINT(l, 3);
      // ---- epilogue: gates and the slice's columns of the new states ----
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int p = tid + e * kFwdThreads;
        if (p >= D::EPI) continue;
        const int i = p / J, j = p % J;
        const int row = t * kTileM + i, hj = hbase + j;
        if (row < r0 || row >= r1) continue;
        float z[D::GATES];
#pragma unroll
        for (int gg = 0; gg < D::GATES; ++gg) {
          const int m = gg * J + j;
          float sum = bias_s[m];
#pragma unroll
          for (int w = 0; w < kFwdWaves; ++w) sum += C_s[(w * 16 + i) * MPAD + m];
          z[gg] = sum;
        }
        const uint32_t el = (uint32_t)(row * H + hj);
        float hv;
        if constexpr (CELL == CORTEX_NARY_TREELSTM) {    // gates (i, f_l, f_r, o, u)
          const float cl = as_float(cc[e][0].x), cr = as_float(cc[e][1].x);
          const float cn = sigmoidf(z[0]) * tanh_f(z[4]) + sigmoidf(z[1]) * cl + sigmoidf(z[2]) * cr;
          hv = sigmoidf(z[3]) * tanh_f(cn);
          cs.store1(el, cn, tag);
          a.c[el] = cn;
        } else {
          hv = tanh_f(z[0]);
        }
        hs.store1(el, hv, tag);
        a.h[el] = hv;
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 4);
      if (tn <= c_last) {
#pragma unroll
        for (int b = 0; b < NB; ++b) fa[b] = fn[b], ea[b] = en[b], ra[b] = rn[b];
#pragma unroll
        for (int e = 0; e < EPT; ++e)
#pragma unroll
          for (int s = 0; s < 2; ++s) cc[e][s] = ccn[e][s], cea[e][s] = cen[e][s];
      }
    }
    }
    CORTEX_TRACE_POINT(l, 5);
    if (load_status(a.status) != 0) return;
  }
  CORTEX_TRACE_KERNEL(3);
}

// ---------------------------------------------------------------------------
// Child-sum TreeLSTM.  Per tile of 16 nodes: the node part x W^T (k split
// over waves 0-3) and the edge part h_k U^T for the 16 x 4 child slots (edge
// tile m = wave & 3, k half = wave >> 2).  The epilogue forms
//   i, o, u = s(W x + sum_k U h_k + b),  f_k = s(W_f x + U_f h_k + b_f),
//   c = i*u + sum_k f_k * c_k,  h = o * tanh(c)
// (U h~ is taken as sum_k U h_k: the same sum in another order).  Child states
// are read from the tagged staging buffers as in the kernel above.
// ---------------------------------------------------------------------------
template <int H, bool kCached>
__global__ void __launch_bounds__(kFwdThreads) childsum_forward_kernel(FwdArgs a) {
  using D = Dims<CORTEX_CHILDSUM_TREELSTM, H>;
  constexpr int J = D::J, LDW = D::LDW, NBX = D::NBX, NBE = D::NBE, KWX = D::KWX, KWE = D::KWE;
  static_assert(D::MPAD == 16 && D::EPI <= kFwdThreads, "one n-tile, one pair per thread");

  __shared__ __attribute__((aligned(16))) float W_s[16 * LDW];
  __shared__ __attribute__((aligned(16))) float C_s[D::C_FLOATS];
  __shared__ float bias_s[16];
  __shared__ ChunkRows chunk;
  extern __shared__ int cache[];
  float *Cx = C_s;                    // [4 waves][16 nodes][16]
  float *Ce = C_s + 4 * 16 * 16;      // [2 halves][64 edges][16]

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int slice = blockIdx.x % a.S, group = blockIdx.x / a.S, Q = a.Q;
  const int hbase = slice * J;
  const int N = a.N, K = a.K;
  const uint32_t tag = a.tag;
  const TagBuf hs(a.hs, (uint32_t)N * H * 8);
  const TagBuf cs(a.cs, (uint32_t)N * H * 8);
  const InBuf xin(a.x_table, (uint32_t)a.x_rows * H * 4);
  const int em = wave & 3, ehalf = wave >> 2;           // edge m-tile and k half of this wave
  const int e_node = (16 * em + i16) >> 2, e_slot = (16 * em + i16) & 3;

  CORTEX_TRACE_KERNEL(0);
  if (load_status(a.status) != 0) return;
  load_weight_slice<CORTEX_CHILDSUM_TREELSTM, H>(a, hbase, W_s, bias_s);
  CORTEX_TRACE_KERNEL(1);
  Structure<kCached> st;
  int L;
  if (!setup_structure<kCached, true, false>(a, cache, st, L)) return;
  CORTEX_TRACE_KERNEL(2);

  for (int l = 0; l < L; ++l) {
    CORTEX_TRACE_POINT(l, 0);
    const int r0 = st.offset(l), r1 = st.offset(l + 1);
    if (!kCached && (r1 < r0 || r1 > N || (l == 0 && r0 != 0))) {
      raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
      return;
    }
    const int t_lo = r0 / kTileM, t_hi = (r1 - 1) / kTileM;
    const int t_first = t_lo + ((group - t_lo % Q) % Q + Q) % Q;

    // structure accessors of the current chunk of tiles
    int c0 = t_first;
    auto child = [&](int t, int i, int s) -> int {
      const int row = t * kTileM + i;
      if (row < r0 || row >= r1 || s >= K) return -1;
      if (kCached) return st.child(row, s);
      return chunk.crow[(t - c0) / Q][i][s];
    };
    auto xrow_of = [&](int t, int i) -> int {
      if (kCached) return st.input_row(t * kTileM + i);
      return chunk.xrow[(t - c0) / Q][i];
    };
    // x fragments (waves 0-3), edge fragments (all waves), children's cells (pairs)
    // every load is issued; absent sources read zeros (no merge, no early wait)
    auto load_tile = [&](int t, u32x4 (&xv)[NBX], Frag4 (&ev)[NBE], int &ecr, u32x2 (&cc)[4],
                         int (&ce)[4]) {
      const int row = t * kTileM + i16;
      int xr = -1;
      if (wave < 4 && row >= r0 && row < r1) xr = xrow_of(t, i16);
#pragma unroll
      for (int b = 0; b < NBX; ++b)
        xv[b] = xin.load4(xr >= 0 ? (uint32_t)((xr * H + wave * KWX + 16 * b + 4 * g4) * 4) : kNoSource);
      ecr = child(t, e_node, e_slot);
#pragma unroll
      for (int b = 0; b < NBE; ++b) {
        const uint32_t off = ecr >= 0 ? (uint32_t)(ecr * H + ehalf * KWE + 16 * b + 4 * g4) * 8u : kNoSource;
        ev[b].lo = hs.load2_at(off);
        ev[b].hi = hs.load2_at(off + 16u);
      }
      const int hj = hbase + tid % J;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int cr = tid < D::EPI ? child(t, tid / J, s) : -1;
        ce[s] = cr >= 0 ? cr * H + hj : -1;
        cc[s] = cs.load1_at(ce[s] >= 0 ? (uint32_t)ce[s] * 8u : kNoSource);
      }
    };

    u32x4 xv[NBX], xn[NBX];
    Frag4 ev[NBE], evn[NBE];
    u32x2 cc[4], ccn[4];
    int ce[4], cen[4];
    int ecr = -1, ecrn = -1;
    for (; c0 <= t_hi; c0 += Q * kChunkTiles) {
    const int c_last = min(t_hi, c0 + Q * (kChunkTiles - 1));
    if (!kCached) {
      __syncthreads();                // the previous chunk's structure is no longer read
      stage_chunk<true, false>(a, chunk, c0, (c_last - c0) / Q + 1, Q, r0, r1);
      __syncthreads();
    }
    load_tile(c0, xv, ev, ecr, cc, ce);
    for (int t = c0; t <= c_last; t += Q) {
      const int tn = t + Q;
      if (tn <= c_last) load_tile(tn, xn, evn, ecrn, ccn, cen);
      CORTEX_TRACE_POINT(l, 1);
      if (ecr >= 0) {
#pragma unroll
        for (int b = 0; b < NBE; ++b) {
          if (!ev[b].staged_ready(tag)) {
            const uint32_t e = (uint32_t)(ecr * H + ehalf * KWE + 16 * b + 4 * g4);
            const uint64_t t0 = wall_clock64();
            int naps = 0;
            do {
              while (hs.load1(e + 3).y != tag && keep_waiting(a.status, t0, a.timeout, naps)) {
              }
              ev[b].lo = hs.load2(e);
              ev[b].hi = hs.load2(e + 2);
            } while (!ev[b].staged_ready(tag) && keep_waiting(a.status, t0, a.timeout, naps));
          }
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
        if (ce[s] >= 0 && cc[s].y != tag) {
          const uint64_t t0 = wall_clock64();
          int naps = 0;
          do {
            cc[s] = cs.load1((uint32_t)ce[s]);
          } while (cc[s].y != tag && keep_waiting(a.status, t0, a.timeout, naps));
        }
      CORTEX_TRACE_POINT(l, 2);
      if (wave < 4) {
        floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
        const float *brow = &W_s[i16 * LDW + wave * KWX + 4 * g4];
#pragma unroll
        for (int b = 0; b < NBX; ++b) {
          const float4 bv = *(const float4 *)(brow + 16 * b);
          if (b & 1) acc1 = mfma_k16(as_float4(xv[b]), bv, acc1);
          else acc0 = mfma_k16(as_float4(xv[b]), bv, acc0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) Cx[(wave * 16 + 4 * g4 + v) * 16 + i16] = acc0[v] + acc1[v];
      }
      {
        floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
        if (__ballot(ecr >= 0) != 0) {      // skip edge tiles with no child at all (leaves)
          const float *brow = &W_s[i16 * LDW + H + ehalf * KWE + 4 * g4];
#pragma unroll
          for (int b = 0; b < NBE; ++b) {
            const float4 bv = *(const float4 *)(brow + 16 * b);
            if (b & 1) acc1 = mfma_k16(ev[b].value(false), bv, acc1);
            else acc0 = mfma_k16(ev[b].value(false), bv, acc0);
          }
        }
#pragma unroll
        for (int v = 0; v < 4; ++v)
          Ce[(ehalf * 64 + 16 * em + 4 * g4 + v) * 16 + i16] = acc0[v] + acc1[v];
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 3);
      if (tid < D::EPI) {
        const int i = tid / J, j = tid % J;
        const int row = t * kTileM + i, hj = hbase + j;
        if (row >= r0 && row < r1) {
          float z[4];       // gate slots (i, o, u, f): x part + bias
#pragma unroll
          for (int gs = 0; gs < 4; ++gs) {
            const int m = gs * J + j;
            z[gs] = bias_s[m] + Cx[(0 * 16 + i) * 16 + m] + Cx[(1 * 16 + i) * 16 + m] +
                    Cx[(2 * 16 + i) * 16 + m] + Cx[(3 * 16 + i) * 16 + m];
          }
          float hs_i = 0.f, hs_o = 0.f, hs_u = 0.f, cpart = 0.f;
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            if (ce[s] >= 0) {
              const float *e0 = &Ce[(0 * 64 + i * 4 + s) * 16];
              const float *e1 = &Ce[(1 * 64 + i * 4 + s) * 16];
              hs_i += e0[0 * J + j] + e1[0 * J + j];
              hs_o += e0[1 * J + j] + e1[1 * J + j];
              hs_u += e0[2 * J + j] + e1[2 * J + j];
              cpart += sigmoidf(z[3] + e0[3 * J + j] + e1[3 * J + j]) * as_float(cc[s].x);
            }
          }
          const float cn = sigmoidf(z[0] + hs_i) * tanh_f(z[2] + hs_u) + cpart;
          const float hv = sigmoidf(z[1] + hs_o) * tanh_f(cn);
          const uint32_t el = (uint32_t)(row * H + hj);
          cs.store1(el, cn, tag);
          hs.store1(el, hv, tag);
          a.c[el] = cn;
          a.h[el] = hv;
        }
      }
      __syncthreads();
      CORTEX_TRACE_POINT(l, 4);
      if (tn <= c_last) {
#pragma unroll
        for (int b = 0; b < NBX; ++b) xv[b] = xn[b];
#pragma unroll
        for (int b = 0; b < NBE; ++b) ev[b] = evn[b];
#pragma unroll
        for (int s = 0; s < 4; ++s) cc[s] = ccn[s], ce[s] = cen[s];
        ecr = ecrn;
      }
    }
    }
    CORTEX_TRACE_POINT(l, 5);
    if (load_status(a.status) != 0) return;
  }
  CORTEX_TRACE_KERNEL(3);
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
// MV-RNN (d = 64): p = tanh(W [B a; A b]), P = W_M [A; B].
// Node-parallel: workgroup b owns output rows [16*(b%4), 16*(b%4)+16) of every
// node it processes (its 16 rows of W and W_M stay in LDS), and node group
// b/4 takes nodes q, q + G/4, ... of each level.  P = W_M[A;B] runs on MFMA
// with [A;B] staged in LDS; the matrix-vector products use VALU.
// ---------------------------------------------------------------------------
constexpr int kMvThreads = 256;
constexpr int kMvD = 64;
constexpr int kMvLd = 2 * kMvD + 4;        // W / W_M slice row stride
constexpr int kMvAb = kMvD + 1;            // [A;B] row stride (odd: row-wise reads spread banks)

__global__ void __launch_bounds__(kMvThreads) mvrnn_forward_kernel(FwdArgs a) {
  constexpr int D = kMvD;
  __shared__ float WM_s[16 * kMvLd];
  __shared__ float Wv_s[16 * kMvLd];
  __shared__ float AB_s[2 * D * kMvAb];
  __shared__ float vec_s[2 * D];          // a (left vector), b (right vector)
  __shared__ float bab_s[2 * D];          // [B a; A b]
  __shared__ int cr_s[2];

  const SyncWords sw{a.sync};
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int rblk = blockIdx.x & 3, ngroup = blockIdx.x >> 2, ngroups = gridDim.x >> 2;
  const DevBuf hb(a.h, (uint32_t)a.N * D * 4);
  const DevBuf pb(a.c, (uint32_t)a.N * D * D * 4);

  bool ok = load_status(a.status) == 0;
  if (!ok) return;
  for (int idx = tid; idx < 16 * 2 * D; idx += kMvThreads) {
    const int r = idx / (2 * D), k = idx % (2 * D);
    WM_s[r * kMvLd + k] = a.W_M[(size_t)(rblk * 16 + r) * 2 * D + k];
    Wv_s[r * kMvLd + k] = a.W[(size_t)(rblk * 16 + r) * 2 * D + k];
  }
  const int L = *a.num_levels;
  if (L < 1 || L > a.N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }
  // leaves: (p, P) = (x_table[x], leaf_mat[x]) or zeros; rows spread over all workgroups
  {
    int r0, r1;
    if (!level_bounds(a, 0, r0, r1)) ok = false;
    for (int r = blockIdx.x; ok && r < r1; r += gridDim.x) {
      const int v = a.level_nodes[r];
      int xi = (v >= 0 && v < a.N) ? a.x_index[v] : -1;
      if (xi < -1 || xi >= a.x_rows) { raise_status(a.status, CORTEX_ST_INPUT_RANGE); xi = -1; }
      if (tid < D / 4) {
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (xi >= 0) val = *(const float4 *)(a.x_table + (size_t)xi * D + tid * 4);
        hb.store4((uint32_t)((r * D + tid * 4) * 4), val);
      }
      for (int e = tid; e < D * D / 4; e += kMvThreads) {
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (xi >= 0) val = *(const float4 *)(a.leaf_mat + (size_t)xi * D * D + e * 4);
        pb.store4((uint32_t)((r * D * D + e * 4) * 4), val);
      }
    }
    if (L > 1) ok = grid_sync<false>(sw, a.status, a.timeout) && ok;
  }
  for (int l = 1; ok && l < L; ++l) {
    int r0, r1;
    if (!level_bounds(a, l, r0, r1)) { ok = false; break; }
    for (int r = r0 + ngroup; r < r1; r += ngroups) {
      if (tid < 2) {
        int cr = a.child_rows[(size_t)r * a.K + tid];
        if (cr < -1 || cr >= r0) { raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION); cr = -1; }
        cr_s[tid] = cr;
      }
      __syncthreads();
      // stage [A; B] (rows 0..63 = A from slot 0, 64..127 = B from slot 1) and a, b
      for (int e = tid; e < 2 * D * D / 4; e += kMvThreads) {
        const int side = e / (D * D / 4), rem = e % (D * D / 4);
        const int rr = rem / (D / 4), c4 = rem % (D / 4);
        const int cr = cr_s[side];
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (cr >= 0) val = pb.load4((uint32_t)((cr * D * D + rr * D + c4 * 4) * 4));
        float *dst = &AB_s[(side * D + rr) * kMvAb + c4 * 4];
        dst[0] = val.x; dst[1] = val.y; dst[2] = val.z; dst[3] = val.w;
      }
      if (tid < 2 * D) {
        const int cr = cr_s[tid / D];
        vec_s[tid] = cr >= 0 ? hb.load1((uint32_t)((cr * D + (tid % D)) * 4)) : 0.f;
      }
      __syncthreads();
      // [B a; A b]: thread k<64 -> (B a)[k] = sum_n B[k][n] a[n];  k>=64 -> (A b)[k-64]
      if (tid < 2 * D) {
        const int k = tid % D;
        const float *mrow = (tid < D) ? &AB_s[(D + k) * kMvAb] : &AB_s[k * kMvAb];
        const float *vv = (tid < D) ? &vec_s[0] : &vec_s[D];
        float s = 0.f;
        for (int n2 = 0; n2 < D; ++n2) s += mrow[n2] * vv[n2];
        bab_s[tid] = s;
      }
      // P rows [16*rblk, +16) = W_M[rows] [A;B]: wave w -> output columns 16w..16w+15
      floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
      for (int k0 = 0; k0 < 2 * D; k0 += 8) {
        acc0 = mfma16x16x4(WM_s[i16 * kMvLd + k0 + g4], AB_s[(k0 + g4) * kMvAb + wave * 16 + i16], acc0);
        acc1 = mfma16x16x4(WM_s[i16 * kMvLd + k0 + 4 + g4], AB_s[(k0 + 4 + g4) * kMvAb + wave * 16 + i16], acc1);
      }
#pragma unroll
      for (int v = 0; v < 4; ++v)
        pb.store1((uint32_t)((r * D * D + (rblk * 16 + 4 * g4 + v) * D + wave * 16 + i16) * 4),
                  acc0[v] + acc1[v]);
      __syncthreads();
      // p rows: 16 outputs x 16 partial sums of 8 terms, reduced over 16 lanes
      {
        const int o = tid >> 4, part = tid & 15;
        float s = 0.f;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) s += Wv_s[o * kMvLd + part * 8 + kk] * bab_s[part * 8 + kk];
        for (int off = 8; off > 0; off >>= 1) s += __shfl_xor(s, off, 16);
        if (part == 0) hb.store1((uint32_t)((r * D + rblk * 16 + o) * 4), tanh_f(s));
      }
      __syncthreads();
    }
    if (l + 1 < L) ok = grid_sync<false>(sw, a.status, a.timeout);
  }
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
typedef void (*KernelFn)(FwdArgs);

struct Instance {
  KernelFn fn;
  int J;
  int threads;
};

constexpr size_t kStructCacheBudget = 40 * 1024;    // bytes of LDS for the cached linearization

// ints of the structure cache: offsets (<= N+1), child rows, input rows, node ids
static size_t cache_ints(int cell, int32_t N, int32_t K) {
  size_t n = (size_t)N + 1 + (size_t)N * K;
  if (cell == CORTEX_TREE_RNN || cell == CORTEX_NARY_TREELSTM || cell == CORTEX_CHILDSUM_TREELSTM) n += N;
  if (cell == CELL_DAG) n += N;
  return n;
}

template <int CELL, int H>
static void pick_slice(bool cached, Instance &out) {
  out.J = Cfg<CELL, H>::J;
  out.threads = kFwdThreads;
  if constexpr (CELL == CORTEX_CHILDSUM_TREELSTM)
    out.fn = cached ? childsum_forward_kernel<H, true> : childsum_forward_kernel<H, false>;
  else
    out.fn = cached ? slice_forward_kernel<CELL, H, true> : slice_forward_kernel<CELL, H, false>;
}

static bool pick(int cell, int H, bool cached, Instance &out) {
#define CORTEX_CASE(CELLID, HH)          \
  if (cell == CELLID && H == HH) {        \
    pick_slice<CELLID, HH>(cached, out);  \
    return true;                          \
  }
  CORTEX_CASE(CORTEX_TREE_RNN, 64)
  CORTEX_CASE(CORTEX_TREE_RNN, 256)
  CORTEX_CASE(CORTEX_NARY_TREELSTM, 64)
  CORTEX_CASE(CORTEX_NARY_TREELSTM, 256)
  CORTEX_CASE(CORTEX_CHILDSUM_TREELSTM, 64)
  CORTEX_CASE(CORTEX_CHILDSUM_TREELSTM, 256)
  CORTEX_CASE(CELL_DAG, 64)
  CORTEX_CASE(CELL_DAG, 256)
#undef CORTEX_CASE
  if (cell == CORTEX_MVRNN && H == kMvD) {
    out.fn = mvrnn_forward_kernel;
    out.J = kMvD;
    out.threads = kMvThreads;
    return true;
  }
  return false;
}

// Workspace of a forward launch: barrier words, the trace area, then the tagged
// staging of h (and of c for the LSTM cells), 8 bytes per element.
static size_t staging_bytes(int32_t N, int32_t H) { return align_up((size_t)N * H * 8, 256); }
static size_t staging_offset() { return align_up(kSyncBytes + kTraceBytes, 256); }
size_t trace_offset() { return kSyncBytes; }
static int staged_tensors(int32_t cell) {
  if (cell == CORTEX_NARY_TREELSTM || cell == CORTEX_CHILDSUM_TREELSTM) return 2;
  if (cell == CORTEX_TREE_RNN || cell == -1) return 1;
  return 0;
}
static std::atomic<uint32_t> g_tag{0};

// A tag no earlier launch used (0 never: a zeroed workspace holds tag 0).
static uint32_t next_tag() {
  uint32_t t = g_tag.fetch_add(1) + 1;
  if (t == 0) t = g_tag.fetch_add(1) + 1;
  return t;
}

static int launch_forward(int cell, int H, const cortex_lin_t *lin, FwdArgs &a, void *d_ws, size_t ws_bytes,
                          void *stream) {
  // state and staging arrays are addressed with 32-bit byte offsets
  const uint64_t state_bytes = (uint64_t)lin->num_nodes * H * (cell == CORTEX_MVRNN ? H : 1) * 8;
  if (state_bytes > 0x7fffffffull) return CORTEX_E_TOO_LARGE;
  if (ws_bytes < cortex_forward_workspace_bytes(cell == CELL_DAG ? -1 : cell, lin->num_nodes, H))
    return CORTEX_E_WORKSPACE;
  size_t dyn = 0;
  bool cached = false;
  if (cell != CORTEX_MVRNN) {
    dyn = cache_ints(cell, lin->num_nodes, lin->max_arity) * sizeof(int);
    cached = dyn <= kStructCacheBudget;
    if (!cached) dyn = 0;
  }
  Instance inst;
  if (!pick(cell, H, cached, inst)) return CORTEX_E_INVAL;
  const int per_cu = cached_occupancy((const void *)inst.fn, inst.threads, dyn);
  const int cus = num_cus();
  if (per_cu <= 0 || cus <= 0) return CORTEX_E_HIP;
  const int cap = per_cu * cus;
  int S;
  int64_t q = knob(CORTEX_KNOB_FWD_NODE_GROUPS);
  if (cell == CORTEX_MVRNN) {
    S = 4;
    if (q <= 0) q = cus / 4;
  } else {
    S = H / inst.J;
    if (q <= 0) q = (S == 1) ? 1 : cus / S;
  }
  if (q < 1) q = 1;
  const int64_t G = S * q;
  if (G > cap || G > kMaxGrid) return CORTEX_E_TOO_LARGE;
  a.S = S;
  a.Q = (int32_t)q;
  a.sync = (unsigned int *)d_ws;
  a.trace = (uint64_t *)((char *)d_ws + kSyncBytes);
  a.timeout = barrier_timeout_ticks();
  const int staged = staged_tensors(cell == CELL_DAG ? -1 : cell);
  char *stage = (char *)d_ws + staging_offset();
  a.hs = staged >= 1 ? stage : nullptr;
  a.cs = staged >= 2 ? stage + staging_bytes(lin->num_nodes, H) : nullptr;
  a.tag = next_tag();
  set_last_grid(1, (int32_t)G);
  return launch_persistent(inst.fn, (int)G, inst.threads, dyn, a, stream);
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
  if (cell < -1 || cell > CORTEX_MVRNN) return 0;
  return cortex::staging_offset() + cortex::staged_tensors(cell) * cortex::staging_bytes(N, H);
}

extern "C" int cortex_tree_forward(int32_t cell, int32_t H, const cortex_lin_t *lin, const float *d_x_table,
                                   int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                                   const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status,
                                   void *d_ws, size_t ws_bytes, void *stream) {
  if (!lin_ok(lin) || !w || !d_status || x_rows < 0) return CORTEX_E_INVAL;
  if (cell < CORTEX_TREE_RNN || cell > CORTEX_MVRNN) return CORTEX_E_INVAL;
  if (lin->num_nodes == 0) return CORTEX_OK;
  if (!d_ws || !d_h || !d_x_index || (x_rows > 0 && !d_x_table)) return CORTEX_E_INVAL;
  const int K = lin->max_arity;
  if (cell == CORTEX_CHILDSUM_TREELSTM) {
    if (!w->W || !w->U || !w->b || !d_c_or_P) return CORTEX_E_INVAL;
  } else {
    if (K != 2) return CORTEX_E_INVAL;
    if (cell == CORTEX_TREE_RNN && (!w->W || !w->b)) return CORTEX_E_INVAL;
    if (cell == CORTEX_NARY_TREELSTM && (!w->U || !w->b || !d_c_or_P)) return CORTEX_E_INVAL;
    if (cell == CORTEX_MVRNN && (!w->W || !w->W_M || !d_c_or_P || (x_rows > 0 && !d_leaf_mat)))
      return CORTEX_E_INVAL;
  }
  FwdArgs a = {};
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
  return launch_forward(cell, H, lin, a, d_ws, ws_bytes, stream);
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
