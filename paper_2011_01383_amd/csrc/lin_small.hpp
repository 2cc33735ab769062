// Linearization of a small batch by one workgroup, entirely in LDS (Sec. 4.2,
// numbering of Appendix B): node heights, level offsets and the stable
// (height, id) row order.  Used by the single-workgroup linearizer kernel and
// by the forward kernels of cortex_tree_infer, where every workgroup
// linearizes the batch for itself before its first level.
#pragma once

#include "cortex_device.hpp"

namespace cortex {

__device__ __forceinline__ int lds_load(const int *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_store(int *p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Exclusive prefix sum of data[0..n) in LDS by the whole workgroup: each
// thread scans a contiguous segment, segment sums are scanned with wave
// shuffles and the wave totals in wsum[THREADS/64 + 1].  Returns the total.
template <int THREADS>
__device__ int block_exclusive_scan(int *data, int n, int *wsum) {
  constexpr int W = THREADS / 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int seg = (n + THREADS - 1) / THREADS;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  int sum = 0;
  for (int i = lo; i < hi; ++i) sum += data[i];
  int x = sum;
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int w = 0; w < W; ++w) {
      const int t = wsum[w];
      wsum[w] = run;
      run += t;
    }
    wsum[W] = run;
  }
  __syncthreads();
  int run = wsum[wave] + x - sum;
  for (int i = lo; i < hi; ++i) {
    const int t = data[i];
    data[i] = run;
    run += t;
  }
  const int total = wsum[W];
  __syncthreads();
  return total;
}

// ---------------------------------------------------------------------------
// Height relaxation over a block of nodes whose heights live in LDS (hs).  A
// thread owns the nodes i = tid + j*THREADS (j < PER; see owned_node for the
// blocked order) and holds their child
// slots in registers: lc = the child's index inside the block (-1 when the
// slot is empty or the child lies outside), ext = a fixed lower bound on the
// height of a child outside the block (-1 otherwise).  A sweep raises h(i) to
// 1 + max over its children.  Values only grow and never pass the true
// height, so sweeps run without barriers, each wave reading whatever the
// others last wrote.  After kSweepBatch such sweeps come a barrier and one
// more sweep: if that sweep changes nothing anywhere, every h(i) equals
// 1 + max over its children as they stand, which is the fixed point, i.e.
// the height.  A value >= N proves a cycle.
// ---------------------------------------------------------------------------
constexpr int kSweepBatch = 4;

// Node j (< PER) of the calling thread: i = tid + j*THREADS, or, with BLK,
// i = tid*PER + j (a thread owns PER consecutive nodes).  wave_has: whether
// some lane of the calling wave owns a node j below n (uniform over the
// wave, and false for every larger j once false).
template <int PER, int THREADS, bool BLK>
__device__ __forceinline__ int owned_node(int j) {
  return BLK ? (int)threadIdx.x * PER + j : (int)threadIdx.x + j * THREADS;
}
template <int PER, int THREADS, bool BLK>
__device__ __forceinline__ bool wave_has(int j, int n) {
  const int wave_first = (int)(threadIdx.x & ~63u);
  return BLK ? wave_first * PER + j < n : wave_first + j * THREADS < n;
}

template <int PER, int THREADS, int KS, bool BLK = false>
__device__ __forceinline__ bool height_sweep(const int (&lc)[PER][4], const int (&ext)[PER][4], int (&myh)[PER],
                                             int *hs, int n, int N, bool &cyc) {
  bool changed = false;
  // A wave reads the child heights of its live nodes back to back, with one
  // wait: whether round j holds live nodes is uniform over the wave, and an
  // empty slot reads entry 0 of the block and is masked.  KS = slots read.
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (!wave_has<PER, THREADS, BLK>(j, n)) break;
    int hv[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) hv[s] = lds_load(&hs[lc[j][s] >= 0 ? lc[j][s] : 0]);
    const int i = owned_node<PER, THREADS, BLK>(j);
    int m = -1;
#pragma unroll
    for (int s = 0; s < KS; ++s) m = max(m, max(lc[j][s] >= 0 ? hv[s] : -1, ext[j][s]));
    if (i < n && m + 1 > myh[j]) {
      myh[j] = m + 1;
      lds_store(&hs[i], m + 1);
      changed = true;
      if (m + 1 >= N) cyc = true;
    }
  }
  return changed;
}

// Dataflow pre-pass before the sweeps: a node's height is computed once,
// when every child it has inside the block is final (hs[c] >= 0; hs holds -1
// for a node not yet computed), as 1 + max over those children and the
// outside lower bounds ext.  Waves run without barriers and each retries its
// pending nodes until all are done, so a chain of dependences advances about
// one node per retry of the wave that holds the next node; a retry requests
// every child height of the thread's nodes at once (one LDS round trip).  A
// cycle (or a very long chain) leaves nodes pending; after max_tries retries
// the pass gives up and leaves them at 0.  Every computed value is the height
// given ext, which is at most the true height, so the sweeps that follow
// start from valid lower bounds and confirm (or finish) the fixed point.
// With BLK (a thread owns consecutive nodes) a height computed in a retry is
// also handed, in registers, to the thread's later nodes that have it as a
// child, so a chain through consecutive ids advances PER nodes per retry.
// Returns (uniformly, after a workgroup barrier) whether every node was
// computed: then the heights are exact for the bounds ext and no sweep can
// change them.
template <int PER, int THREADS, int KS, bool BLK = false>
__device__ bool height_dataflow(const int (&lc)[PER][4], const int (&ext)[PER][4], int (&myh)[PER], int *hs, int n,
                                int max_tries) {
  // per node: the LDS slots of its in-block children (absent ones read slot
  // 0, masked out below) and the bound from the children outside the block
  int slot[PER][KS], ebound[PER];
  unsigned inmask[PER];
  bool pending[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    pending[j] = owned_node<PER, THREADS, BLK>(j) < n;
    inmask[j] = 0u;
    ebound[j] = -1;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      slot[j][s] = lc[j][s] >= 0 ? lc[j][s] : 0;
      inmask[j] |= lc[j][s] >= 0 ? 1u << s : 0u;
      ebound[j] = max(ebound[j], ext[j][s]);
    }
  }
  for (int tries = 0; tries < max_tries; ++tries) {
    bool left = false;
    int hvs[PER][KS];
#pragma unroll
    for (int j = 0; j < PER; ++j)
#pragma unroll
      for (int s = 0; s < KS; ++s) hvs[j][s] = lds_load(&hs[slot[j][s]]);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (!wave_has<PER, THREADS, BLK>(j, n)) break;
      // an in-block child that is not final yet (-1) keeps the node pending
      int m = ebound[j];
      unsigned wait = 0u;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bool in = (inmask[j] >> s) & 1u;
        m = max(m, in ? hvs[j][s] : -1);
        wait |= (in && hvs[j][s] < 0) ? 1u : 0u;
      }
      const bool fire = pending[j] && wait == 0u;
      if (fire) {
        const int i = owned_node<PER, THREADS, BLK>(j);
        myh[j] = m + 1;
        lds_store(&hs[i], m + 1);
        if constexpr (BLK) {
#pragma unroll
          for (int j2 = j + 1; j2 < PER; ++j2)
#pragma unroll
            for (int s = 0; s < KS; ++s)
              if (((inmask[j2] >> s) & 1u) && slot[j2][s] == i) hvs[j2][s] = m + 1;
        }
      }
      pending[j] = pending[j] && !fire;
      left = left || pending[j];
    }
    if (!__any(left)) break;
  }
  bool any_left = false;
#pragma unroll
  for (int j = 0; j < PER; ++j) any_left = any_left || (owned_node<PER, THREADS, BLK>(j) < n && pending[j]);
  const bool complete = !__syncthreads_or(any_left);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = owned_node<PER, THREADS, BLK>(j);
    if (i < n && pending[j]) {
      myh[j] = 0;
      lds_store(&hs[i], 0);
    }
  }
  __syncthreads();
  return complete;
}

// Sweeps to the fixed point over child slots [0, KS).  Returns (uniformly
// over the workgroup) whether any height changed; *cycle is set when a value
// reached N.  Every thread of the workgroup calls it.
template <int PER, int THREADS, int KS, bool BLK = false>
__device__ bool relax_heights_k(const int (&lc)[PER][4], const int (&ext)[PER][4], int (&myh)[PER], int *hs, int n,
                                int N, bool *cycle, int *sweeps) {
  bool any = false;
  *cycle = false;
  for (;;) {
    bool cyc = false;
#pragma unroll 1
    for (int r = 0; r < kSweepBatch; ++r) any |= height_sweep<PER, THREADS, KS, BLK>(lc, ext, myh, hs, n, N, cyc);
    __syncthreads();
    const bool ch = height_sweep<PER, THREADS, KS, BLK>(lc, ext, myh, hs, n, N, cyc);
    any |= ch;
    *sweeps += kSweepBatch + 1;
    if (__syncthreads_or(cyc)) {
      *cycle = true;
      break;
    }
    if (!__syncthreads_or(ch)) break;
  }
  return __syncthreads_or(any) != 0;
}

template <int PER, int THREADS, bool BLK = false>
__device__ bool relax_heights(const int (&lc)[PER][4], const int (&ext)[PER][4], int (&myh)[PER], int *hs, int n,
                              int K, int N, bool *cycle, int *sweeps) {
  if (K <= 2) return relax_heights_k<PER, THREADS, 2, BLK>(lc, ext, myh, hs, n, N, cycle, sweeps);
  return relax_heights_k<PER, THREADS, 4, BLK>(lc, ext, myh, hs, n, N, cycle, sweeps);
}

// ---------------------------------------------------------------------------
// One workgroup of THREADS threads linearizes N <= THREADS * PER nodes:
//   children -> LDS; heights (a forest, where every node fills at most one
//   child slot, by a last-arriver walk from the leaves; any other DAG by
//   height sweeps until nothing changes, a value >= N proving a cycle); a
//   stable counting sort on height with 8-bit digits (one pass while L <=
//   256): a global digit histogram gives each digit's first row, then
//   THREADS-node chunks in id order are ranked with wave ballots, per-wave
//   digit counts and a running cursor per digit.
// LDS (ints, small_lin_ints): children N*K, height N, perm 2N, node_row N,
// level count N+1, wave-digit counts (THREADS/64)*256, digit cursors 256*2,
// 64 of scratch.
// ---------------------------------------------------------------------------
template <int THREADS>
__host__ __device__ constexpr size_t small_lin_ints(int N, int K) {
  return (size_t)N * K + 5 * (size_t)N + 1 + (size_t)(THREADS / 64) * 256 + 2 * 256 + 64;
}

// Results in LDS: ch[v*K+s] the validated child slots, hgt[v] the height of
// node v, order[r] the node of row r, nrow[v] the row of node v and
// lcount[l] the first row of level l (l < L).
struct SmallLin {
  const int *ch, *hgt, *nrow, *lcount, *order;
};

// Trace builds: stamps[k] = the wall clock at phase k (thread 0), when given.
#ifdef CORTEX_TRACE
#define LIN_STAMP(k)                                             \
  do {                                                           \
    if (stamps && threadIdx.x == 0) stamps[(k)] = wall_clock64(); \
  } while (0)
#else
#define LIN_STAMP(k) \
  do {               \
  } while (0)
#endif

// ---------------------------------------------------------------------------
// Batches of at most 64 * kWavePer nodes: wave 0 linearizes alone, with no
// workgroup barrier (the others wait at one).  One wave's LDS operations are
// performed in program order, so a value one lane stores is what any lane
// of the wave loads afterwards; compiler fences keep that order.  Node v
// sits in lane v % 64, slot v / 64.
//   heights  rounds of h(v) = 1 + max over its children (0 for a leaf), all
//            nodes in every round, until a round changes nothing: values only
//            grow and never pass the true height, so the fixed point is the
//            height; a value >= N proves a cycle;
//   offsets  level counts by LDS atomics, then an exclusive scan by the wave
//            in chunks of 64 levels;
//   rows     slots in order (ids ascending); within a slot the lanes of one
//            height are matched by ballots on the height's bits and ranked by
//            lane, after the rows already taken in that level (a cursor per
//            level): the stable (height, id) order.
// Same LDS layout and results as the multi-wave path below.
// ---------------------------------------------------------------------------
constexpr int kWavePer = 2;

template <int THREADS, int KS>
__device__ int wave_linearize(const int32_t *children, int N, int K, int32_t *status, int status0, int *sm,
                              SmallLin &m, uint64_t *stamps) {
  (void)stamps;
  const int tid = threadIdx.x, lane = tid & 63;
  int *ch = sm;                       // [N*K]
  int *hgt = ch + N * K;              // [N]
  int *perm0 = hgt + N;               // [N]  row -> node
  int *perm1 = perm0 + N;             // [N]  level cursors
  int *nrow = perm1 + N;              // [N]
  int *lcount = nrow + N;             // [N+1]
  int *flags = lcount + N + 1 + (THREADS / 64) * 256 + 2 * 256;   // [64] scratch
  if (tid < 64) {
    int myc[kWavePer][KS], myh[kWavePer];
#pragma unroll
    for (int p = 0; p < kWavePer; ++p)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int v = lane + 64 * p;
        myc[p][s] = children[(v < N && s < K) ? (size_t)v * K + s : 0];
      }
    int bad = 0;
#pragma unroll
    for (int p = 0; p < kWavePer; ++p) {
      const int v = lane + 64 * p;
      myh[p] = 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        int c = (v < N && s < K) ? myc[p][s] : -1;
        if (c < -1 || c >= N) { bad = 1; c = -1; }
        myc[p][s] = c;
        if (v < N && s < K) lds_store(&ch[v * K + s], c);
      }
      if (v < N) {
        lds_store(&hgt[v], 0);
        lds_store(&lcount[v], 0);
      }
    }
    LIN_STAMP(1);
    int err = __shfl(status0, 0) != 0 ? -1 : (__ballot(bad) != 0ull ? CORTEX_ST_CHILD_RANGE : 0);
    int L = 0;
    const int nslots = (N + 63) >> 6;
    if (err == 0) {
      for (;;) {
        // a round: every child height is requested first, then every node
        // updated, so the round costs one LDS round trip
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        int hv[kWavePer][KS];
#pragma unroll
        for (int p = 0; p < kWavePer; ++p)
          if (p < nslots) {
#pragma unroll
            for (int s = 0; s < KS; ++s) hv[p][s] = lds_load(&hgt[myc[p][s] >= 0 ? myc[p][s] : 0]);
          }
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        bool changed = false, cyc = false;
#pragma unroll
        for (int p = 0; p < kWavePer; ++p) {
          const int v = lane + 64 * p;
          if (p >= nslots) break;
          int mx = -1;
#pragma unroll
          for (int s = 0; s < KS; ++s) mx = max(mx, myc[p][s] >= 0 ? hv[p][s] : -1);
          if (v < N && mx + 1 > myh[p]) {
            myh[p] = mx + 1;
            lds_store(&hgt[v], mx + 1);
            changed = true;
            if (mx + 1 >= N) cyc = true;
          }
        }
        if (__ballot(cyc) != 0ull) {
          err = CORTEX_ST_CYCLE;
          break;
        }
        if (__ballot(changed) == 0ull) break;
      }
    }
    LIN_STAMP(2);
    if (err == 0) {
      int mx = 0;
#pragma unroll
      for (int p = 0; p < kWavePer; ++p)
        if (lane + 64 * p < N) mx = max(mx, myh[p]);
      for (int off = 32; off > 0; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
      L = mx + 1;
      // level counts (lcount was cleared above, by this wave)
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
#pragma unroll
      for (int p = 0; p < kWavePer; ++p)
        if (lane + 64 * p < N)
          __hip_atomic_fetch_add(&lcount[myh[p]], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      // exclusive scan into lcount (level offsets) and perm1 (cursors)
      int carry = 0;
      for (int base = 0; base < L; base += 64) {
        const int l = base + lane;
        const int cnt = l < L ? lds_load(&lcount[l]) : 0;
        int x = cnt;
        for (int off = 1; off < 64; off <<= 1) {
          const int y = __shfl_up(x, off);
          if (lane >= off) x += y;
        }
        if (l < L) {
          lds_store(&lcount[l], carry + x - cnt);
          lds_store(&perm1[l], carry + x - cnt);
        }
        carry += __shfl(x, 63);
      }
      LIN_STAMP(3);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      const int nbits = 32 - __clz(L - 1);                      // bits of the largest height
      const unsigned long long lt_mask = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
#pragma unroll
      for (int p = 0; p < kWavePer; ++p) {
        const int v = lane + 64 * p;
        if (p >= nslots) break;
        const bool valid = v < N;
        const int dig = valid ? myh[p] : 0;
        unsigned long long peers = __ballot(valid);
        for (int b = 0; b < nbits; ++b) {
          const bool bit = (dig >> b) & 1;
          const unsigned long long mb = __ballot(bit);
          peers &= bit ? mb : ~mb;
        }
        const int base = lds_load(&perm1[dig]);                // every lane reads before any writes
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        const int row = base + __popcll(peers & lt_mask);
        if (valid) {
          if ((peers & lt_mask) == 0ull) lds_store(&perm1[dig], base + __popcll(peers));
          lds_store(&perm0[row], v);
          lds_store(&nrow[v], row);
        }
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
      }
      LIN_STAMP(4);
    }
    if (lane == 0) {
      flags[0] = err == 0 ? L : 0;
      flags[1] = err;
    }
  }
  __syncthreads();
  const int L = flags[0], err = flags[1];
  if (err > 0) {
    if (tid == 0) raise_status(status, err);
    return 0;
  }
  if (err != 0) return 0;
  m.ch = ch;
  m.hgt = hgt;
  m.nrow = nrow;
  m.lcount = lcount;
  m.order = perm0;
  return L;
}

// Returns L >= 1, or 0 (uniformly) after raising a status: a child index out
// of range, a cycle, or a non-zero status on entry.
template <int THREADS, int PER>
__device__ int small_linearize(const int32_t *children, int N, int K, int32_t *status, int *sm, SmallLin &m,
                               uint64_t *stamps) {
  constexpr int WAVES = THREADS / 64;
  (void)stamps;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int *ch = sm;                       // [N*K]
  int *hgt = ch + N * K;              // [N]
  int *perm0 = hgt + N;               // [N]
  int *perm1 = perm0 + N;             // [N]
  int *nrow = perm1 + N;              // [N]
  int *lcount = nrow + N;             // [N+1]
  int *wcnt = lcount + N + 1;         // [16][256]
  int *dstart = wcnt + WAVES * 256;   // [256]
  int *cursor = dstart + 256;         // [256]
  int *flags = cursor + 256;          // [64] scratch

  LIN_STAMP(0);
  const int status0 = load_status(status);     // requested together with the children
  if (N <= 64 * kWavePer)
    return K <= 2 ? wave_linearize<THREADS, 2>(children, N, K, status, status0, sm, m, stamps)
                  : wave_linearize<THREADS, 4>(children, N, K, status, status0, sm, m, stamps);
  // 1. children: into registers for the sweeps (node v = tid + j*threads) and
  //    into LDS for the output phase; range check
  int myc[PER][4], myh[PER];
  int bad = 0;
  // every load is issued before any result is used (an absent slot reads
  // entry 0 and is masked), so they cost one memory round trip together
#pragma unroll
  for (int j = 0; j < PER; ++j)
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int v = tid + j * THREADS;
      myc[j][s] = children[(v < N && s < K) ? (size_t)v * K + s : 0];
    }
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int v = tid + j * THREADS;
    myh[j] = 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      int c = (v < N && s < K) ? myc[j][s] : -1;
      if (c < -1 || c >= N) { bad = 1; c = -1; }
      myc[j][s] = c;
      if (v < N && s < K) ch[v * K + s] = c;
    }
    if (v < N) hgt[v] = 0;
  }
  if (__syncthreads_or(status0 != 0)) return 0;
  if (__syncthreads_or(bad)) {
    if (tid == 0) raise_status(status, CORTEX_ST_CHILD_RANGE);
    return 0;
  }
  LIN_STAMP(1);
  // 2. heights.  Forest (every node fills at most one child slot in the
  //    whole batch): a last-arriver walk.  Each node counts its pending
  //    children; the thread of a leaf climbs towards the root: at each
  //    parent it raises the parent's height to its own + 1, then takes one
  //    off the parent's count, and the thread that empties the count holds
  //    the parent's final height and climbs on.  A node still pending
  //    afterwards lies on or above a cycle.  Any other DAG: barrier-free
  //    sweeps to the fixed point.  (perm0, nrow and lcount serve as the
  //    parent-count, parent and pending arrays here; all are rewritten later.)
  //    The walk's LDS operations stay in program order (compiler fences) and
  //    the LDS unit performs one wave's operations in that order, so the
  //    raise lands before the decrement and the last decrement sees every
  //    sibling's raise.
  int *npar = perm0, *parent = nrow, *pend = lcount;
  int multi = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int v = tid + j * THREADS;
    if (v < N) {
      npar[v] = 0;
      parent[v] = -1;
      pend[v] = (myc[j][0] >= 0) + (myc[j][1] >= 0) + (myc[j][2] >= 0) + (myc[j][3] >= 0);
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int v = tid + j * THREADS;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int c = myc[j][s];
      if (c >= 0) {
        // a second parent of c is seen by the thread whose increment finds 1
        if (__hip_atomic_fetch_add(&npar[c], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0) multi = 1;
        parent[c] = v;
      }
    }
  }
  if (!__syncthreads_or(multi)) {
#pragma unroll 1
    for (int j = 0; j < PER; ++j) {
      const int v = tid + j * THREADS;
      if (v >= N || (myc[j][0] >= 0) + (myc[j][1] >= 0) + (myc[j][2] >= 0) + (myc[j][3] >= 0) != 0) continue;
      int hu = 0, p = parent[v];
      while (p >= 0) {
        __hip_atomic_fetch_max(&hgt[p], hu + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        const int left = __hip_atomic_fetch_sub(&pend[p], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (left != 1) break;
        hu = lds_load(&hgt[p]);
        p = lds_load(&parent[p]);
      }
    }
    __syncthreads();
    int stuck = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int v = tid + j * THREADS;
      if (v < N) {
        if (pend[v] != 0) stuck = 1;
        myh[j] = hgt[v];
      }
    }
    if (__syncthreads_or(stuck)) {
      if (tid == 0) raise_status(status, CORTEX_ST_CYCLE);
      return 0;
    }
  } else {
    int ext[PER][4];
#pragma unroll
    for (int j = 0; j < PER; ++j)
#pragma unroll
      for (int s = 0; s < 4; ++s) ext[j][s] = -1;
    // dataflow order first (hgt = -1: not computed), then sweeps confirm
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (tid + j * THREADS < N) lds_store(&hgt[tid + j * THREADS], -1);
    __syncthreads();
    if (K <= 2)
      height_dataflow<PER, THREADS, 2>(myc, ext, myh, hgt, N, 4 * N);
    else
      height_dataflow<PER, THREADS, 4>(myc, ext, myh, hgt, N, 4 * N);
    bool cyc;
    int sweeps = 0;
    relax_heights<PER, THREADS>(myc, ext, myh, hgt, N, K, N, &cyc, &sweeps);
    if (cyc) {
      if (tid == 0) raise_status(status, CORTEX_ST_CYCLE);
      return 0;
    }
  }
  LIN_STAMP(2);
  // L = 1 + max height, level counts
  int mx = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) mx = max(mx, myh[j]);
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, __shfl_xor(mx, off));
  if (lane == 0) flags[wave] = mx;
  for (int i = tid; i <= N; i += THREADS) lcount[i] = 0;
  __syncthreads();
  int L = 0;
  for (int w = 0; w < WAVES; ++w) L = max(L, flags[w]);
  L += 1;
  for (int v = tid; v < N; v += THREADS) atomicAdd(&lcount[hgt[v]], 1);
  __syncthreads();
  // level offsets = exclusive scan of the level counts (kept in lcount): by
  // wave 0 alone up to 64 levels, else by the whole workgroup
  if (L <= 64) {
    if (tid < 64) {
      const int cnt = tid < L ? lcount[tid] : 0;
      int x = cnt;
      for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      if (tid < L) lcount[tid] = x - cnt;
    }
    __syncthreads();
  } else {
    block_exclusive_scan<THREADS>(lcount, L, flags);
  }
  LIN_STAMP(3);
  // 3. stable LSD counting sort on height, 8-bit digits.  With one pass
  //    (L <= 256) the digit is the height itself: its starts are the level
  //    offsets, and only bits(L-1) ballots and L digit columns are needed.
  int passes = 1;
  for (int v = (L - 1) >> 8; v > 0; v >>= 8) ++passes;
  const int nbits = passes == 1 ? 32 - __clz(L - 1) : 8;      // __clz(0) = 32: L = 1 needs none
  const int ndig = passes == 1 ? L : 256;
  const unsigned long long lt_mask = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    const int *in = (p & 1) ? perm0 : perm1;    // pass 0 reads ids directly
    int *out = (p & 1) ? perm1 : perm0;
    if (passes == 1) {
      if (tid < L) dstart[tid] = lcount[tid];
    } else {
      if (tid < 256) dstart[tid] = 0;
      __syncthreads();
      for (int i = tid; i < N; i += THREADS) {
        const int v = p == 0 ? i : in[i];
        atomicAdd(&dstart[(hgt[v] >> shift) & 255], 1);
      }
      __syncthreads();
      block_exclusive_scan<THREADS>(dstart, 256, flags);
    }
    if (tid < 256) cursor[tid] = 0;
    __syncthreads();
    for (int base = 0; base < N; base += THREADS) {
      const int idx = base + tid;
      const bool valid = idx < N;
      const int item = valid ? (p == 0 ? idx : in[idx]) : 0;
      const int dig = valid ? ((hgt[item] >> shift) & 255) : 0;
      unsigned long long peers = __ballot(valid);
      for (int b = 0; b < nbits; ++b) {
        const bool bit = (dig >> b) & 1;
        const unsigned long long m = __ballot(bit);
        peers &= bit ? m : ~m;
      }
      const int rank = __popcll(peers & lt_mask);
      for (int i = tid; i < WAVES * ndig; i += THREADS) wcnt[(i / ndig) * 256 + i % ndig] = 0;
      __syncthreads();
      if (valid && rank == 0) wcnt[wave * 256 + dig] = __popcll(peers);
      __syncthreads();
      if (tid < ndig) {            // per digit: wave offsets within the chunk, then advance the cursor
        int run = cursor[tid];
        for (int w = 0; w < WAVES; ++w) { const int x = wcnt[w * 256 + tid]; wcnt[w * 256 + tid] = run; run += x; }
        cursor[tid] = run;
      }
      __syncthreads();
      if (valid) out[dstart[dig] + wcnt[wave * 256 + dig] + rank] = item;
      __syncthreads();
    }
  }
  LIN_STAMP(4);
  const int *order = ((passes - 1) & 1) ? perm1 : perm0;
  for (int r = tid; r < N; r += THREADS) nrow[order[r]] = r;
  __syncthreads();
  m.ch = ch;
  m.hgt = hgt;
  m.nrow = nrow;
  m.lcount = lcount;
  m.order = order;
  return L;
}

// Writes the linearization (cortex_lin_t arrays) from the LDS results; every
// thread of the workgroup takes part.
template <int THREADS>
__device__ void small_lin_emit(const SmallLin &m, int N, int K, int L, int32_t *num_levels, int32_t *height,
                               int32_t *level_offsets, int32_t *level_nodes, int32_t *node_row,
                               int32_t *child_rows) {
  const int tid = threadIdx.x;
  for (int l = tid; l < L; l += THREADS) level_offsets[l] = m.lcount[l];
  if (tid == 0) {
    level_offsets[L] = N;
    *num_levels = L;
  }
  for (int r = tid; r < N; r += THREADS) {
    const int v = m.order[r];
    level_nodes[r] = v;
    node_row[v] = r;
    height[r] = m.hgt[r];             // by node id (r doubles as a node id here)
    for (int s = 0; s < K; ++s) {
      const int c = m.ch[v * K + s];
      child_rows[(size_t)r * K + s] = c < 0 ? -1 : m.nrow[c];
    }
  }
}

}  // namespace cortex
