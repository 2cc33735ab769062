// Data-structure linearization on the GPU (Sec. 4.2, numbering of Appendix B).
//
// One persistent cooperative kernel computes, for N nodes of arity K:
//   1. heights: height(v) = 0 without children, else 1 + max over children.
//      Each workgroup owns a contiguous chunk of node ids held in LDS and
//      relaxes it to a local fixed point (children outside the chunk are read
//      from HBM); global rounds repeat until no workgroup changes a height.
//      Values only grow and never exceed the true height, so the fixed point
//      is the height; a value >= N proves a cycle.
//   2. rows: a stable least-significant-digit counting sort of the node ids
//      on height (8-bit digits, one pass while L <= 256).  Each pass builds
//      per-tile digit histograms, scans them in (digit, tile) order and
//      scatters every tile with wave-ballot ranking, which keeps equal keys
//      in id order.  The result is the dynamic-batching order: level by level,
//      ascending id inside a level.
//   3. level offsets from the height steps along the sorted rows, and the
//      child rows through node_row.
#include "cortex_device.hpp"
#include "cortex_host.hpp"
#include "lin_small.hpp"

namespace cortex {

constexpr int kLinThreads = 1024;
// The digit phases of the sort give thread t < 256 digit t: the per-tile
// histograms, the digit bases and their scan index 256-entry arrays (and the
// global tile histograms) by thread id, so every such access sits behind
// `digit_thread`; threads 256 and up only join the barriers there.
constexpr int kDigits = 256;
static_assert(kLinThreads >= kDigits && kLinThreads % 64 == 0, "a thread per 8-bit digit");
constexpr int kLinWaves = kLinThreads / 64;
constexpr int kTile = 1024;                  // radix tile
constexpr int kSubs = kTile / 64;            // 64-item sub-chunks per tile
constexpr int kSubsPerWave = kSubs / kLinWaves;
constexpr int kMaxChunk = 8192;              // heights per workgroup held in LDS
constexpr int kTargetChunk = 1024;           // default chunk when the grid is free
constexpr int kLinPer = kTargetChunk / kLinThreads;   // nodes per thread whose children sit in registers


struct LinArgs {
  const int32_t *children;
  int32_t N, K;
  int32_t *num_levels, *height, *level_offsets, *level_nodes, *node_row, *child_rows;
  int32_t *status;
  unsigned int *sync;
  int32_t *tile_hist;          // [256 * tiles]
  int32_t *perm_a, *perm_b;    // [N] ping-pong between sort passes
  int32_t chunk, tiles;
  uint64_t timeout;
};


// Maximum over the workgroup (tmp: kLinThreads ints of LDS); every thread gets it.
__device__ __forceinline__ int block_max(int v, int *tmp) {
  for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = v;
  __syncthreads();
  int m = tmp[0];
  for (int w = 1; w < kLinWaves; ++w) m = max(m, tmp[w]);
  __syncthreads();
  return m;
}


// Trace builds only: workgroup 0 stamps phase boundaries into uint64 slots
// 1..15 of the barrier header (the generation word uses slot 0 only).
#ifdef CORTEX_TRACE
#define CORTEX_BIG_STAMP(k, v)                                                        \
  do {                                                                               \
    if (blockIdx.x == 0 && threadIdx.x == 0) ((uint64_t *)a.sync)[(k)] = (v);          \
  } while (0)
#else
#define CORTEX_BIG_STAMP(k, v) \
  do {                         \
  } while (0)
#endif

// kDual: compiled for two workgroups per compute unit (8 waves per SIMD, 64
// VGPRs, a few spilled), the instance for batches of more radix tiles than
// one workgroup per compute unit can hold one tile each.
template <bool kDual>
__global__ void __launch_bounds__(kLinThreads, kDual ? 8 : 1) linearize_kernel(LinArgs a) {
  __shared__ int hs[kMaxChunk];
  __shared__ int cnt[kSubs][256];
  __shared__ int hist[256];
  __shared__ int base_s[256];
  __shared__ int scan_tmp[kLinThreads];

  const SyncWords sw{a.sync};
  const int tid = threadIdx.x;
  const bool digit_thread = tid < kDigits;
  const int G = gridDim.x;
  const int N = a.N, K = a.K;
  const int lo = blockIdx.x * a.chunk;
  const int hi = min(N, lo + a.chunk);
  const int n = max(0, hi - lo);
  CORTEX_BIG_STAMP(1, wall_clock64());
  const int status0 = load_status(a.status);     // requested together with the children
  int sweeps0 = 0;

  // ---------------- 1. heights ----------------
  // The children of a chunk of at most kLinPer nodes per thread (the default
  // chunk) go to registers once, thread t holding nodes kLinPer*t ..
  // kLinPer*t + kLinPer - 1; a larger chunk reads them on every sweep.
  const bool in_regs = n <= kLinPer * kLinThreads;
  int cid[kLinPer][4], lc[kLinPer][4], ext[kLinPer][4], myh[kLinPer];
  int bad = 0;
  // all loads issued before any is used (absent slots read entry 0, masked)
#pragma unroll
  for (int j = 0; j < kLinPer; ++j)
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int i = owned_node<kLinPer, kLinThreads, true>(j);
      cid[j][s] = a.children[(in_regs && i < n && s < K) ? (size_t)(lo + i) * K + s : 0];
    }
#pragma unroll
  for (int j = 0; j < kLinPer; ++j) {
    const int i = owned_node<kLinPer, kLinThreads, true>(j);
    myh[j] = 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      int c = (in_regs && i < n && s < K) ? cid[j][s] : -1;
      if (c < -1 || c >= N) {
        bad = 1;
        c = -1;
      }
      cid[j][s] = c;
      lc[j][s] = (c >= lo && c < hi) ? c - lo : -1;
      ext[j][s] = -1;
    }
  }
  bool ok = status0 == 0;
  if (bad) raise_status(a.status, CORTEX_ST_CHILD_RANGE);
  for (int i = tid; i < n; i += kLinThreads) hs[i] = in_regs ? -1 : 0;
  __syncthreads();
  CORTEX_BIG_STAMP(9, wall_clock64());
  bool complete0 = false;
  if (in_regs && ok) {
    // round 0: children outside the chunk count 0 (a lower bound); nodes
    // whose in-chunk children are final are computed once, in dataflow order
#pragma unroll
    for (int j = 0; j < kLinPer; ++j)
#pragma unroll
      for (int s = 0; s < 4; ++s) ext[j][s] = (cid[j][s] < 0 || lc[j][s] >= 0) ? -1 : 0;
    if (K <= 2)
      complete0 = height_dataflow<kLinPer, kLinThreads, 2, true>(lc, ext, myh, hs, n, 4 * kTargetChunk);
    else
      complete0 = height_dataflow<kLinPer, kLinThreads, 4, true>(lc, ext, myh, hs, n, 4 * kTargetChunk);
  }
  CORTEX_BIG_STAMP(10, wall_clock64());
  // a chunk whose children all lie inside it reaches its exact heights in
  // round 0; only when some chunk reads an outside child (counted 0 in round
  // 0) does a second round have to check the fixed point across chunks
  int has_ext = 0;
  if (in_regs) {
#pragma unroll
    for (int j = 0; j < kLinPer; ++j)
#pragma unroll
      for (int s = 0; s < 4; ++s) has_ext |= (cid[j][s] >= 0 && lc[j][s] < 0);
  } else {
    has_ext = 1;
  }
  has_ext = __syncthreads_or(has_ext);
  const int T = a.tiles;
  // every workgroup's chunk is its radix tile: the sort then reads heights
  // from LDS, gets its first histograms from the height rounds, and the
  // child rows are written per node
  const bool own_tile = a.chunk == kTile && G == T && in_regs;
  int round = 0;
  int L = 0;
  while (ok) {
    int block_changed = (round == 0) && has_ext;
    int local_max = 0;
    if (in_regs) {
      // children outside the chunk keep one height per round: 0 in round 0
      // (a lower bound), then what the previous round published
#pragma unroll
      for (int j = 0; j < kLinPer; ++j)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int c = cid[j][s];
          ext[j][s] = (c < 0 || lc[j][s] >= 0)
                          ? -1
                          : (round == 0 ? 0 : __hip_atomic_load(&a.height[c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        }
      bool cyc = false;
      // (round 0 reports has_ext alone: a chunk without outside children
      // is exact whatever its sweeps changed.  When the dataflow pass
      // computed every node, round 0 needs no sweep at all.)
      if (!(round == 0 && complete0) &&
          relax_heights<kLinPer, kLinThreads, true>(lc, ext, myh, hs, n, K, N, &cyc, &sweeps0) && round > 0)
        block_changed = 1;
      if (cyc && tid == 0) raise_status(a.status, CORTEX_ST_CYCLE);
    } else for (;;) {
      int changed = 0, cyc = 0;
      for (int i = tid; i < n; i += kLinThreads) {
        const int v = lo + i;
        int m = -1;
        for (int s = 0; s < K; ++s) {
          int c = a.children[(size_t)v * K + s];
          if (c < -1 || c >= N) {
            if (round == 0) raise_status(a.status, CORTEX_ST_CHILD_RANGE);
            continue;
          }
          if (c < 0) continue;
          int hc;
          if (c >= lo && c < hi) hc = lds_load(&hs[c - lo]);
          else if (round == 0) hc = 0;    // global heights not written yet: 0 is a lower bound
          else hc = __hip_atomic_load(&a.height[c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          m = max(m, hc);
        }
        const int nh = m + 1;
        if (nh > lds_load(&hs[i])) {
          lds_store(&hs[i], nh);
          changed = 1;
          if (nh >= N) {
            raise_status(a.status, CORTEX_ST_CYCLE);
            cyc = 1;
          }
        }
      }
      // uniform exit decision for the whole workgroup
      const int any = __syncthreads_or(changed);
      const int stop = __syncthreads_or(cyc);
      if (round == 0) ++sweeps0;
      block_changed |= any;
      if (!any || stop) break;
    }
    for (int i = tid; i < n; i += kLinThreads) {
      const int hv = hs[i];
      __hip_atomic_store(&a.height[lo + i], hv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      local_max = max(local_max, hv);
    }
    local_max = block_max(local_max, scan_tmp);
    if (own_tile) {
      // the first sort pass's digit histogram of this tile, from this
      // round's heights; after the last round they are final, and the grid
      // barrier below publishes the histogram with them
      if (digit_thread) hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < n; i += kLinThreads) atomicAdd(&hist[hs[i] & 255], 1);
      __syncthreads();
      if (digit_thread) a.tile_hist[(size_t)tid * T + blockIdx.x] = hist[tid];
    }
    if (round == 0) CORTEX_BIG_STAMP(11, wall_clock64());
    if (G == 1) {
      L = local_max + 1;
      ok = grid_sync(sw, a.status, a.timeout);
      break;                                      // one chunk: the local fixed point is global
    }
    // publish (changed, max) in this round's parity slot, then combine all of them
    if (tid == 0) {
      st_agent(sw.slot(0, round & 1, blockIdx.x), (unsigned)block_changed);
      st_agent(sw.slot(1, round & 1, blockIdx.x), (unsigned)local_max);
    }
    ok = grid_sync(sw, a.status, a.timeout);
    if (round == 0) CORTEX_BIG_STAMP(12, wall_clock64());
    if (!ok) break;
    int any = 0, mx = 0;
    for (int b = tid; b < G; b += kLinThreads) {
      any |= (int)ld_agent(sw.slot(0, round & 1, b));
      mx = max(mx, (int)ld_agent(sw.slot(1, round & 1, b)));
    }
    any = __syncthreads_or(any);
    mx = block_max(mx, scan_tmp);
    ++round;
    if (!any) {
      L = mx + 1;
      break;
    }
  }

  CORTEX_BIG_STAMP(2, wall_clock64());
  CORTEX_BIG_STAMP(7, (uint64_t)round);
  CORTEX_BIG_STAMP(8, (uint64_t)sweeps0);
  // ---------------- 2. stable counting sort on height ----------------
  int passes = 1;
  for (int v = (L - 1) >> 8; v > 0; v >>= 8) ++passes;
  const bool rows_per_node = own_tile && passes == 1;
  // every child lies in its parent's chunk (round 0 found no chunk reading
  // outside itself, so the height loop stopped after it, or there is one
  // chunk): a chunk's child rows then come from its own rows in LDS, and no
  // barrier across workgroups is needed after the scatter
  const bool rows_local = rows_per_node && (G == 1 || round == 1);
  const int wave = tid >> 6, lane = tid & 63;
  const unsigned long long lt_mask = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));

  for (int p = 0; ok && p < passes; ++p) {
    const int shift = 8 * p;
    const int32_t *in = (p == 0) ? nullptr : ((p & 1) ? a.perm_a : a.perm_b);
    const bool last = (p == passes - 1);
    int32_t *out = last ? a.level_nodes : ((p & 1) ? a.perm_b : a.perm_a);

    // (a) per-tile digit histograms, stored digit-major (those of the first
    //     pass already came with the heights when every chunk is a tile)
    for (int t = blockIdx.x; t < T && !(own_tile && p == 0); t += G) {
      if (digit_thread) hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < kTile; i += kLinThreads) {
        const int idx = t * kTile + i;
        if (idx < N) {
          const int item = in ? in[idx] : idx;
          atomicAdd(&hist[(a.height[item] >> shift) & 255], 1);
        }
      }
      __syncthreads();
      if (digit_thread) a.tile_hist[(size_t)tid * T + t] = hist[tid];
      __syncthreads();
    }
    if (!(own_tile && p == 0)) ok = grid_sync(sw, a.status, a.timeout);
    if (!ok) break;
    if (p == 0) CORTEX_BIG_STAMP(3, wall_clock64());

    // (c) stable scatter: rank = (digit base of this tile) + (equal digits
    //     earlier in the tile).  Sub-chunk q of 64 items goes to wave
    //     q / kSubsPerWave.
    for (int t = blockIdx.x; t < T; t += G) {
      // digit bases of tile t, from every tile's histogram: the rows of all
      // smaller digits, plus the rows of the same digit in earlier tiles
      {
        int tot = 0, before = 0;
        if (!digit_thread) {
          // no digit: only the scan's barriers
        } else if ((T & 3) == 0 && ((uintptr_t)a.tile_hist & 15) == 0) {
          // this digit's row of T counts, 16 bytes per load, all in flight
          const int4 *row = (const int4 *)(a.tile_hist + (size_t)tid * T);
#pragma unroll 16
          for (int t4 = 0; t4 < T / 4; ++t4) {
            const int4 x = row[t4];
            const int b = 4 * t4;
            tot += x.x + x.y + x.z + x.w;
            before += (b < t ? x.x : 0) + (b + 1 < t ? x.y : 0) + (b + 2 < t ? x.z : 0) + (b + 3 < t ? x.w : 0);
          }
        } else {
#pragma unroll 32
          for (int t2 = 0; t2 < T; ++t2) {
            const int x = a.tile_hist[(size_t)tid * T + t2];
            tot += x;
            before += t2 < t ? x : 0;
          }
        }
        if (digit_thread) hist[tid] = tot;
        __syncthreads();
        block_exclusive_scan<kLinThreads>(hist, kDigits, scan_tmp);
        if (digit_thread) base_s[tid] = hist[tid] + before;
        // one pass: digit = height, so a digit's first row is its level's
        if (rows_per_node && blockIdx.x == 0 && digit_thread && tid < L) a.level_offsets[tid] = hist[tid];
      }
      if (p == 0 && t == (int)blockIdx.x) CORTEX_BIG_STAMP(4, wall_clock64());
      for (int i = tid; i < kSubs * 256; i += kLinThreads) (&cnt[0][0])[i] = 0;
      __syncthreads();
      int item[kSubsPerWave], dig[kSubsPerWave], rank[kSubsPerWave];
      bool valid[kSubsPerWave];
#pragma unroll
      for (int qq = 0; qq < kSubsPerWave; ++qq) {
        const int q = wave * kSubsPerWave + qq;
        const int idx = t * kTile + q * 64 + lane;
        valid[qq] = idx < N;
        item[qq] = valid[qq] ? (in ? in[idx] : idx) : 0;
        const int hq = !valid[qq] ? 0 : (own_tile && p == 0) ? hs[idx - lo] : a.height[item[qq]];
        dig[qq] = (hq >> shift) & 255;
        unsigned long long peers = __ballot(valid[qq]);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const bool bit = (dig[qq] >> b) & 1;
          const unsigned long long m = __ballot(bit);
          peers &= bit ? m : ~m;
        }
        rank[qq] = __popcll(peers & lt_mask);
        if (valid[qq] && rank[qq] == 0) cnt[q][dig[qq]] = __popcll(peers);
      }
      __syncthreads();
      if (digit_thread) {   // exclusive scan over sub-chunks, one digit per thread
        int run = 0;
        for (int q = 0; q < kSubs; ++q) { int x = cnt[q][tid]; cnt[q][tid] = run; run += x; }
      }
      __syncthreads();
#pragma unroll
      for (int qq = 0; qq < kSubsPerWave; ++qq) {
        if (!valid[qq]) continue;
        const int q = wave * kSubsPerWave + qq;
        const int pos = base_s[dig[qq]] + cnt[q][dig[qq]] + rank[qq];
        if (pos < 0 || pos >= N) {              // cannot happen for consistent counts
          raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
          continue;
        }
        out[pos] = item[qq];
        if (last) a.node_row[item[qq]] = pos;
        if (rows_per_node) hs[kTile + q * 64 + lane] = pos;     // this chunk's node q*64 + lane
      }
      __syncthreads();
    }
    if (!(last && rows_local)) ok = grid_sync(sw, a.status, a.timeout);
  }
  CORTEX_BIG_STAMP(5, wall_clock64());

  // ---------------- 3. level offsets and child rows ----------------
  if (ok && rows_per_node) {
    // per node of this chunk: its row (kept in LDS by the scatter) and its
    // child slots (in registers) give its child rows; a child's row is in
    // LDS too when it lies in the chunk and every child does (rows_local),
    // else its chunk wrote it before the barrier above.  (The level offsets
    // came from the digit starts.)
    int pos[kLinPer], cr[kLinPer][4];
#pragma unroll
    for (int j = 0; j < kLinPer; ++j) {
      const int i = owned_node<kLinPer, kLinThreads, true>(j);
      pos[j] = i < n ? hs[kTile + i] : -1;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int c = (i < n && s < K) ? cid[j][s] : -1;
        cr[j][s] = c < 0 ? -1 : (rows_local && lc[j][s] >= 0) ? hs[kTile + lc[j][s]] : a.node_row[c];
      }
    }
#pragma unroll
    for (int j = 0; j < kLinPer; ++j)
      if (pos[j] >= 0 && pos[j] < N)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (s < K) a.child_rows[(size_t)pos[j] * K + s] = cr[j][s];
    if (blockIdx.x == 0 && tid == 0) {
      a.level_offsets[L] = N;
      *a.num_levels = L;
    }
  } else if (ok) {
    const int gtid = blockIdx.x * kLinThreads + tid;
    const int gstride = G * kLinThreads;
    for (int r = gtid; r < N; r += gstride) {
      const int h = a.height[a.level_nodes[r]];
      const int hp = r > 0 ? a.height[a.level_nodes[r - 1]] : -1;
      for (int l = hp + 1; l <= h; ++l) a.level_offsets[l] = r;
      const int v = a.level_nodes[r];
      for (int s = 0; s < K; ++s) {
        const int c = a.children[(size_t)v * K + s];
        a.child_rows[(size_t)r * K + s] = c < 0 ? -1 : a.node_row[c];
      }
    }
    if (blockIdx.x == 0 && tid == 0) {
      a.level_offsets[L] = N;
      *a.num_levels = L;
    }
  }
  CORTEX_BIG_STAMP(6, wall_clock64());
}


// ---------------------------------------------------------------------------
// Small batches: one workgroup does the whole linearization in LDS
// (small_linearize), then writes every output array once, coalesced.
// ---------------------------------------------------------------------------
constexpr int kSmallThreads = 1024;
constexpr int kSmallPer = 4;                         // nodes per thread: N <= 4096
constexpr size_t kSmallLdsMax = 150 * 1024;

static size_t small_lds_bytes(int32_t N, int32_t K) { return sizeof(int) * small_lin_ints<kSmallThreads>(N, K); }


__global__ void __launch_bounds__(kSmallThreads) linearize_small_kernel(LinArgs a) {
  extern __shared__ int sm[];
  SmallLin m;
  uint64_t *stamps = nullptr;
#ifdef CORTEX_TRACE
  stamps = (uint64_t *)a.sync;
#endif
  const int L = small_linearize<kSmallThreads, kSmallPer>(a.children, a.N, a.K, a.status, sm, m, stamps);
  if (L == 0) return;
  small_lin_emit<kSmallThreads>(m, a.N, a.K, L, a.num_levels, a.height, a.level_offsets, a.level_nodes,
                                a.node_row, a.child_rows);
  LIN_STAMP(5);
  LIN_STAMP(6);
}

static size_t lin_tiles(int32_t N) { return (size_t)(N + kTile - 1) / kTile; }

__global__ void write_zero_kernel(int32_t *p) { *p = 0; }

}  // namespace cortex

using namespace cortex;

extern "C" size_t cortex_linearize_workspace_bytes(int32_t N, int32_t K) {
  if (N < 0 || K < 1 || K > 4) return 0;
  size_t b = kSyncBytes;
  b += align_up(256 * lin_tiles(N) * sizeof(int32_t), 256);
  b += 2 * align_up((size_t)N * sizeof(int32_t), 256);
  return b;
}

namespace cortex {

// dry_run: every host check of the call, nothing enqueued.
int linearize_impl(const int32_t *d_children, int32_t N, int32_t K, const cortex_lin_t *lin, int32_t *d_status,
                   void *d_ws, size_t ws_bytes, void *stream, bool dry_run) {
  if (!lin || !d_status || N < 0 || K < 1 || K > 4) return CORTEX_E_INVAL;
  if (lin->num_nodes != N || lin->max_arity != K || !lin->num_levels) return CORTEX_E_INVAL;
  if (N == 0) {
    if (dry_run) return CORTEX_OK;
    // an empty batch has no levels; a one-lane kernel (not a memset node, so
    // the call can be captured into a graph) writes L = 0
    int32_t *p = lin->num_levels;
    void *kargs[] = {(void *)&p};
    return hipLaunchKernel((const void *)write_zero_kernel, dim3(1), dim3(1), kargs, 0, (hipStream_t)stream) ==
                   hipSuccess
               ? CORTEX_OK
               : CORTEX_E_HIP;
  }
  if (!d_children || !lin->height || !lin->level_offsets || !lin->level_nodes || !lin->node_row ||
      !lin->child_rows || !d_ws)
    return CORTEX_E_INVAL;
  if (ws_bytes < cortex_linearize_workspace_bytes(N, K)) return CORTEX_E_WORKSPACE;

  const size_t small_lds = small_lds_bytes(N, K);
  if (knob(CORTEX_KNOB_LIN_BLOCKS) == 0 && small_lds <= kSmallLdsMax && N <= kSmallThreads * kSmallPer) {
    LinArgs s = {};
    s.children = d_children;
    s.N = N;
    s.K = K;
    s.num_levels = lin->num_levels;
    s.height = lin->height;
    s.level_offsets = lin->level_offsets;
    s.level_nodes = lin->level_nodes;
    s.node_row = lin->node_row;
    s.child_rows = lin->child_rows;
    s.status = d_status;
    s.sync = (unsigned int *)d_ws;
    if (cached_occupancy((const void *)linearize_small_kernel, kSmallThreads, small_lds) <= 0) return CORTEX_E_HIP;
    if (dry_run) return CORTEX_OK;
    set_last_grid(0, 1);
    return launch_persistent(linearize_small_kernel, 1, kSmallThreads, small_lds, s, stream);
  }
  int cap = max_coresident(linearize_kernel<false>, kLinThreads);
  if (cap <= 0) return CORTEX_E_HIP;
  int64_t g = knob(CORTEX_KNOB_LIN_BLOCKS);
  // one radix tile per workgroup keeps every node's children in registers:
  // where one workgroup per compute unit cannot give each tile its own, the
  // two-per-unit instance can (up to twice as many tiles)
  bool dual = false;
  if (g <= 0) {
    g = (N + kTargetChunk - 1) / kTargetChunk;
    if (g > cap && g <= kMaxGrid) {
      const int cap2 = max_coresident(linearize_kernel<true>, kLinThreads);
      if (g <= cap2) {
        dual = true;
        cap = cap2;
      }
    }
  }
  const int64_t g_min = (N + kMaxChunk - 1) / kMaxChunk;
  if (g < g_min) g = g_min;
  if (g > N) g = N;
  if (cap > kMaxGrid) cap = kMaxGrid;
  if (g > cap) {
    if (g_min > cap) return CORTEX_E_TOO_LARGE;
    g = cap;
  }
  if (dry_run) return CORTEX_OK;
  LinArgs a;
  a.children = d_children;
  a.N = N;
  a.K = K;
  a.num_levels = lin->num_levels;
  a.height = lin->height;
  a.level_offsets = lin->level_offsets;
  a.level_nodes = lin->level_nodes;
  a.node_row = lin->node_row;
  a.child_rows = lin->child_rows;
  a.status = d_status;
  char *ws = (char *)d_ws;
  a.sync = (unsigned int *)ws;
  ws += kSyncBytes;
  a.tiles = (int32_t)lin_tiles(N);
  a.tile_hist = (int32_t *)ws;
  ws += align_up(256 * (size_t)a.tiles * sizeof(int32_t), 256);
  a.perm_a = (int32_t *)ws;
  ws += align_up((size_t)N * sizeof(int32_t), 256);
  a.perm_b = (int32_t *)ws;
  // one chunk per radix tile when the grid has one workgroup per tile
  a.chunk = g == (int64_t)a.tiles ? kTile : (int32_t)((N + g - 1) / g);
  a.timeout = barrier_timeout_ticks();
  set_last_grid(0, (int32_t)g);
  return dual ? launch_persistent(linearize_kernel<true>, (int)g, kLinThreads, 0, a, stream)
              : launch_persistent(linearize_kernel<false>, (int)g, kLinThreads, 0, a, stream);
}

}  // namespace cortex

extern "C" int cortex_linearize(const int32_t *d_children, int32_t N, int32_t K, const cortex_lin_t *lin,
                                int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream) {
  return linearize_impl(d_children, N, K, lin, d_status, d_ws, ws_bytes, stream, false);
}
