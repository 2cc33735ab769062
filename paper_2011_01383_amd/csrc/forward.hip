// Persistent level-synchronous forward kernels (Sec. 4.1 loop nest; kernel
// fusion and model persistence as evaluated in Sec. 7.2-7.3).
//
// One cooperative launch runs every level.  Workgroup b owns hidden slice
// s = b % S (J hidden units, all gates of those units) and node group
// q = b / S.  Its slice of the cell weights is loaded into LDS once and stays
// there for the whole pass (persistence).  Per level, the level's rows are cut
// into 16-row tiles and group q takes tiles q, q+Q, ...; for each tile the
// workgroup gathers the child state rows (and inputs) into LDS, contracts them
// with its weight slice on the fp32 MFMA units, applies the gate
// nonlinearities in registers and writes its J columns of the new states.
// A device-wide barrier separates levels (the dependence is carried by the
// level loop only, Appendix A.4).  The leaf level of TreeRNN, N-ary TreeLSTM
// and MV-RNN is a specialised copy (Sec. 3.1 specialization, Sec. 4.3 zero
// initial state).
#include "cortex_device.hpp"
#include "cortex_host.hpp"

namespace cortex {

constexpr int kFwdThreads = 256;
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kTileM = 16;
constexpr int CELL_DAG = 16;                 // internal id of the DAG-RNN cell

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
  static constexpr int LDW = KA + 4;                       // padded row stride (bank spread)
  static constexpr bool kChildSum = CELL == CORTEX_CHILDSUM_TREELSTM;
  static constexpr int LDX = H + 4;
  // generic: A tile [16][LDW]; child-sum: x tile [16][LDX] + edge tile [64][LDX]
  static constexpr int A_FLOATS = kChildSum ? (16 + 64) * LDX : 16 * LDW;
  // generic: per-wave partials [4][16][MPAD]; child-sum: Cx [4][16][16] + Ce [64][16]
  static constexpr int C_FLOATS = kChildSum ? (4 * 16 * 16 + 64 * 16) : 4 * 16 * MPAD;
  static_assert(KA % (4 * 16) == 0, "k range per wave must be a multiple of 16");
  static_assert(H % J == 0, "slices must tile H");
};

// Row of the resident weight slice for (gate slot g, unit j) and its bias.
// Child-sum rows are ordered (i, o, u, f); the input layout is (i, f, o, u).
__device__ __forceinline__ int childsum_gate(int gslot) {
  return gslot == 0 ? 0 : (gslot == 1 ? 2 : (gslot == 2 ? 3 : 1));
}

template <int CELL, int H>
__device__ void load_weight_slice(const FwdArgs &a, int hbase, float *W_s, float *bias_s) {
  using D = Dims<CELL, H>;
  constexpr int F4 = D::KA / 4, SEG4 = H / 4;
  for (int idx = threadIdx.x; idx < D::MPAD * F4; idx += kFwdThreads) {
    const int m = idx / F4, c4 = idx % F4;
    const int g = m / D::J, j = m % D::J, hj = hbase + j;
    const int sg = c4 / SEG4, o4 = c4 % SEG4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (m < D::GATES * D::J) {
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

// Leaf level of TreeRNN / N-ary TreeLSTM: h = x_table[x_index[node]] (or 0),
// c = 0.  Rows are spread over all workgroups, one float4 per thread.
template <int H>
__device__ void leaf_copy(const FwdArgs &a, int r1, bool with_c) {
  constexpr int F4 = H / 4;
  constexpr int ROWS = kFwdThreads / F4 > 0 ? kFwdThreads / F4 : 1;
  const int sub = threadIdx.x / F4, c4 = threadIdx.x % F4;
  if (sub >= ROWS) return;
  for (int r = blockIdx.x * ROWS + sub; r < r1; r += gridDim.x * ROWS) {
    const int v = a.level_nodes[r];
    int xi = (v >= 0 && v < a.N) ? a.x_index[v] : -1;
    if (xi < -1 || xi >= a.x_rows) {
      raise_status(a.status, CORTEX_ST_INPUT_RANGE);
      xi = -1;
    }
    float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
    if (xi >= 0) val = *(const float4 *)(a.x_table + (size_t)xi * H + c4 * 4);
    *(float4 *)(a.h + (size_t)r * H + c4 * 4) = val;
    if (with_c) *(float4 *)(a.c + (size_t)r * H + c4 * 4) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

template <int CELL, int H>
__global__ void __launch_bounds__(kFwdThreads) slice_forward_kernel(FwdArgs a) {
  using D = Dims<CELL, H>;
  constexpr int J = D::J, MPAD = D::MPAD, NT = D::NT, LDW = D::LDW, LDX = D::LDX;
  constexpr int KA = D::KA;
  constexpr int SLOTS = D::kChildSum ? 4 : (CELL == CELL_DAG ? 2 : 2);

  __shared__ __attribute__((aligned(16))) float W_s[MPAD * LDW];
  __shared__ __attribute__((aligned(16))) float A_s[D::A_FLOATS];
  __shared__ __attribute__((aligned(16))) float C_s[D::C_FLOATS];
  __shared__ float bias_s[MPAD];
  __shared__ int cr_s[kTileM][4];
  __shared__ int node_s[kTileM];

  const SyncWords sw{a.sync};
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int slice = blockIdx.x % a.S, group = blockIdx.x / a.S;
  const int hbase = slice * J;

  bool ok = load_status(a.status) == 0;
  if (!ok) return;

  load_weight_slice<CELL, H>(a, hbase, W_s, bias_s);
  __syncthreads();

  const int L = *a.num_levels;
  if (L < 1 || L > a.N) {
    raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
    return;
  }

  int first = 0;
  if (CELL == CORTEX_TREE_RNN || CELL == CORTEX_NARY_TREELSTM) {
    int r0, r1;
    if (!level_bounds(a, 0, r0, r1)) ok = false;
    else leaf_copy<H>(a, r1, CELL == CORTEX_NARY_TREELSTM);
    first = 1;
    if (L > 1) ok = grid_sync(sw, a.status, a.timeout) && ok;
  }

  for (int l = first; ok && l < L; ++l) {
    int r0, r1;
    if (!level_bounds(a, l, r0, r1)) { ok = false; break; }
    const int tiles = (r1 - r0 + kTileM - 1) / kTileM;
    for (int t = group; t < tiles; t += a.Q) {
      const int rb = r0 + t * kTileM;
      const int nv = min(kTileM, r1 - rb);
      // ---- stage node ids and validated child rows of the tile ----
      if (tid < kTileM * 4) {
        const int i = tid >> 2, sl = tid & 3;
        int cr = -1;
        if (i < nv && sl < SLOTS && sl < a.K) {
          cr = a.child_rows[(size_t)(rb + i) * a.K + sl];
          if (cr < -1 || cr >= r0) {             // a child must sit in a lower level
            raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION);
            cr = -1;
          }
        }
        cr_s[i][sl] = cr;
      }
      if (tid < kTileM) {
        int v = tid < nv ? a.level_nodes[rb + tid] : -1;
        if (v < -1 || v >= a.N) { raise_status(a.status, CORTEX_ST_BAD_LINEARIZATION); v = -1; }
        node_s[tid] = v;
      }
      __syncthreads();

      if constexpr (!D::kChildSum) {
        // ---- gather the A tile: [h(slot0) | h(slot1)] or [x | h(slot0) | h(slot1)] ----
        constexpr int F4 = KA / 4, SEG4 = H / 4;
        for (int idx = tid; idx < kTileM * F4; idx += kFwdThreads) {
          const int i = idx / F4, c4 = idx % F4, sg = c4 / SEG4, o4 = c4 % SEG4;
          const float *src = nullptr;
          if (i < nv) {
            if (CELL == CELL_DAG) {
              if (sg == 0) { const int v = node_s[i]; if (v >= 0) src = a.x + (size_t)v * H; }
              else { const int cr = cr_s[i][sg - 1]; if (cr >= 0) src = a.h + (size_t)cr * H; }
            } else {
              const int cr = cr_s[i][sg];
              if (cr >= 0) src = a.h + (size_t)cr * H;
            }
          }
          float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
          if (src) v = *(const float4 *)(src + o4 * 4);
          *(float4 *)&A_s[i * LDW + c4 * 4] = v;
        }
        __syncthreads();

        // ---- contraction: wave w covers k in [w*KA/4, (w+1)*KA/4) ----
        constexpr int KW = KA / kFwdWaves;
        floatx4 acc0[NT], acc1[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc0[nt] = acc1[nt] = floatx4{0.f, 0.f, 0.f, 0.f};
        const float *arow = &A_s[i16 * LDW + wave * KW + 4 * g4];
        const float *brow = &W_s[i16 * LDW + wave * KW + 4 * g4];
        // two independent accumulator chains (k blocks of 16 alternate)
        for (int kb = 0; kb + 32 <= KW; kb += 32) {
          const float4 a0 = *(const float4 *)(arow + kb);
          const float4 a1 = *(const float4 *)(arow + kb + 16);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const float4 b0 = *(const float4 *)(brow + nt * 16 * LDW + kb);
            const float4 b1 = *(const float4 *)(brow + nt * 16 * LDW + kb + 16);
            acc0[nt] = mfma_k16(a0, b0, acc0[nt]);
            acc1[nt] = mfma_k16(a1, b1, acc1[nt]);
          }
        }
        if constexpr (KW % 32 == 16) {
          const int kb = KW - 16;
          const float4 a0 = *(const float4 *)(arow + kb);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            acc0[nt] = mfma_k16(a0, *(const float4 *)(brow + nt * 16 * LDW + kb), acc0[nt]);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            C_s[(wave * 16 + 4 * g4 + v) * MPAD + nt * 16 + i16] = acc0[nt][v] + acc1[nt][v];
        __syncthreads();

        // ---- epilogue: gates and state write for (row i, unit j) ----
        for (int p = tid; p < kTileM * J; p += kFwdThreads) {
          const int i = p / J, j = p % J;
          if (i >= nv) continue;
          const size_t row = (size_t)(rb + i);
          const int hj = hbase + j;
          float z[D::GATES];
#pragma unroll
          for (int gg = 0; gg < D::GATES; ++gg) {
            const int m = gg * J + j;
            float s = bias_s[m];
#pragma unroll
            for (int w = 0; w < kFwdWaves; ++w) s += C_s[(w * 16 + i) * MPAD + m];
            z[gg] = s;
          }
          if constexpr (CELL == CORTEX_TREE_RNN || CELL == CELL_DAG) {
            a.h[row * H + hj] = tanh_f(z[0]);
          } else {   // N-ary: gates (i, f_l, f_r, o, u)
            const int cl = cr_s[i][0], cr = cr_s[i][1];
            const float c_l = cl >= 0 ? a.c[(size_t)cl * H + hj] : 0.f;
            const float c_r = cr >= 0 ? a.c[(size_t)cr * H + hj] : 0.f;
            const float cn = sigmoidf(z[0]) * tanh_f(z[4]) + sigmoidf(z[1]) * c_l + sigmoidf(z[2]) * c_r;
            a.c[row * H + hj] = cn;
            a.h[row * H + hj] = sigmoidf(z[3]) * tanh_f(cn);
          }
        }
        __syncthreads();
      } else {
        // ---- child-sum: x tile [16][H] and edge tile [16 nodes x 4 slots][H] ----
        float *X_s = A_s;
        float *E_s = A_s + 16 * LDX;
        float *Cx = C_s;                  // [4 waves][16][16]
        float *Ce = C_s + 4 * 16 * 16;    // [64 edges][16]
        constexpr int F4 = H / 4;
        for (int idx = tid; idx < 80 * F4; idx += kFwdThreads) {
          const int r = idx / F4, c4 = idx % F4;
          const float *src = nullptr;
          if (r < 16) {
            const int v = node_s[r];
            if (v >= 0) {
              int xi = a.x_index[v];
              if (xi < -1 || xi >= a.x_rows) { raise_status(a.status, CORTEX_ST_INPUT_RANGE); xi = -1; }
              if (xi >= 0) src = a.x_table + (size_t)xi * H;
            }
          } else {
            const int e = r - 16;
            const int cr = cr_s[e >> 2][e & 3];
            if (cr >= 0) src = a.h + (size_t)cr * H;
          }
          float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
          if (src) v = *(const float4 *)(src + c4 * 4);
          *(float4 *)&A_s[r * LDX + c4 * 4] = v;
        }
        __syncthreads();
        // node part, k split over waves: Cx[w] = x[:, kq] W^T[kq, :]
        {
          constexpr int KW = H / kFwdWaves;
          floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
          const float *arow = &X_s[i16 * LDX + wave * KW + 4 * g4];
          const float *brow = &W_s[i16 * LDW + wave * KW + 4 * g4];
          for (int kb = 0; kb + 32 <= KW; kb += 32) {
            acc0 = mfma_k16(*(const float4 *)(arow + kb), *(const float4 *)(brow + kb), acc0);
            acc1 = mfma_k16(*(const float4 *)(arow + kb + 16), *(const float4 *)(brow + kb + 16), acc1);
          }
          if constexpr (KW % 32 == 16)
            acc0 = mfma_k16(*(const float4 *)(arow + KW - 16), *(const float4 *)(brow + KW - 16), acc0);
#pragma unroll
          for (int v = 0; v < 4; ++v) Cx[(wave * 16 + 4 * g4 + v) * 16 + i16] = acc0[v] + acc1[v];
        }
        // edge part: wave w takes edge rows 16w..16w+15 (nodes 4w..4w+3), all k: Ce = h_e U^T
        if (l > 0) {
          floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
          const float *arow = &E_s[(wave * 16 + i16) * LDX + 4 * g4];
          const float *brow = &W_s[i16 * LDW + H + 4 * g4];
          for (int kb = 0; kb < H; kb += 32) {      // H is a multiple of 32
            acc0 = mfma_k16(*(const float4 *)(arow + kb), *(const float4 *)(brow + kb), acc0);
            acc1 = mfma_k16(*(const float4 *)(arow + kb + 16), *(const float4 *)(brow + kb + 16), acc1);
          }
#pragma unroll
          for (int v = 0; v < 4; ++v) Ce[(wave * 16 + 4 * g4 + v) * 16 + i16] = acc0[v] + acc1[v];
        }
        __syncthreads();
        for (int p = tid; p < kTileM * J; p += kFwdThreads) {
          const int i = p / J, j = p % J;
          if (i >= nv) continue;
          const size_t row = (size_t)(rb + i);
          const int hj = hbase + j;
          float z[4];     // slots (i, o, u, f): x part + bias
#pragma unroll
          for (int gs = 0; gs < 4; ++gs) {
            const int m = gs * J + j;
            z[gs] = bias_s[m] + Cx[(0 * 16 + i) * 16 + m] + Cx[(1 * 16 + i) * 16 + m] +
                    Cx[(2 * 16 + i) * 16 + m] + Cx[(3 * 16 + i) * 16 + m];
          }
          float cn_parts[4];
          float hs_i = 0.f, hs_o = 0.f, hs_u = 0.f;
#pragma unroll
          for (int sl = 0; sl < 4; ++sl) {
            const int cr = cr_s[i][sl];
            cn_parts[sl] = 0.f;
            if (cr >= 0) {
              const float *ce = &Ce[(i * 4 + sl) * 16];
              hs_i += ce[0 * J + j];
              hs_o += ce[1 * J + j];
              hs_u += ce[2 * J + j];
              const float f = sigmoidf(z[3] + ce[3 * J + j]);
              cn_parts[sl] = f * a.c[(size_t)cr * H + hj];
            }
          }
          float cn = sigmoidf(z[0] + hs_i) * tanh_f(z[2] + hs_u);
#pragma unroll
          for (int sl = 0; sl < 4; ++sl) cn += cn_parts[sl];
          a.c[row * H + hj] = cn;
          a.h[row * H + hj] = sigmoidf(z[1] + hs_o) * tanh_f(cn);
        }
        __syncthreads();
      }
    }
    if (l + 1 < L) ok = grid_sync(sw, a.status, a.timeout);
  }
}

// ---------------------------------------------------------------------------
// MV-RNN (d = 64): p = tanh(W [B a; A b]), P = W_M [A; B].
// Node-parallel: workgroup b owns output rows [16*(b%4), 16*(b%4)+16) of every
// node it processes (its 16 rows of W and W_M stay in LDS), and node group
// b/4 takes nodes q, q + G/4, ... of each level.  P = W_M[A;B] runs on MFMA
// with [A;B] staged in LDS; the matrix-vector products use VALU.
// ---------------------------------------------------------------------------
constexpr int kMvD = 64;
constexpr int kMvLd = 2 * kMvD + 4;        // W / W_M slice row stride
constexpr int kMvAb = kMvD + 1;            // [A;B] row stride (odd: row-wise reads spread banks)

__global__ void __launch_bounds__(kFwdThreads) mvrnn_forward_kernel(FwdArgs a) {
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

  bool ok = load_status(a.status) == 0;
  if (!ok) return;
  for (int idx = tid; idx < 16 * 2 * D; idx += kFwdThreads) {
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
        *(float4 *)(a.h + (size_t)r * D + tid * 4) = val;
      }
      for (int e = tid; e < D * D / 4; e += kFwdThreads) {
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (xi >= 0) val = *(const float4 *)(a.leaf_mat + (size_t)xi * D * D + e * 4);
        *(float4 *)(a.c + (size_t)r * D * D + e * 4) = val;
      }
    }
    if (L > 1) ok = grid_sync(sw, a.status, a.timeout) && ok;
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
      for (int e = tid; e < 2 * D * D / 4; e += kFwdThreads) {
        const int side = e / (D * D / 4), rem = e % (D * D / 4);
        const int rr = rem / (D / 4), c4 = rem % (D / 4);
        const int cr = cr_s[side];
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (cr >= 0) val = *(const float4 *)(a.c + (size_t)cr * D * D + rr * D + c4 * 4);
        float *dst = &AB_s[(side * D + rr) * kMvAb + c4 * 4];
        dst[0] = val.x; dst[1] = val.y; dst[2] = val.z; dst[3] = val.w;
      }
      if (tid < 2 * D) {
        const int cr = cr_s[tid / D];
        vec_s[tid] = cr >= 0 ? a.h[(size_t)cr * D + (tid % D)] : 0.f;
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
        a.c[(size_t)r * D * D + (size_t)(rblk * 16 + 4 * g4 + v) * D + wave * 16 + i16] = acc0[v] + acc1[v];
      __syncthreads();
      // p rows: 16 outputs x 16 partial sums of 8 terms, reduced over 16 lanes
      {
        const int o = tid >> 4, part = tid & 15;
        float s = 0.f;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) s += Wv_s[o * kMvLd + part * 8 + kk] * bab_s[part * 8 + kk];
        for (int off = 8; off > 0; off >>= 1) s += __shfl_xor(s, off, 16);
        if (part == 0) a.h[(size_t)r * D + rblk * 16 + o] = tanh_f(s);
      }
      __syncthreads();
    }
    if (l + 1 < L) ok = grid_sync(sw, a.status, a.timeout);
  }
}

// ---------------------------------------------------------------------------
// Host dispatch
// ---------------------------------------------------------------------------
typedef void (*KernelFn)(FwdArgs);

struct Instance {
  KernelFn fn;
  int J;
};

static bool pick(int cell, int H, Instance &out) {
#define CORTEX_CASE(CELLID, HH)                                        \
  if (cell == CELLID && H == HH) {                                      \
    out.fn = slice_forward_kernel<CELLID, HH>;                          \
    out.J = Cfg<CELLID, HH>::J;                                         \
    return true;                                                        \
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
    return true;
  }
  return false;
}

static int launch_forward(int cell, int H, const cortex_lin_t *lin, FwdArgs &a, void *d_ws, size_t ws_bytes,
                          void *stream) {
  Instance inst;
  if (!pick(cell, H, inst)) return CORTEX_E_INVAL;
  if (ws_bytes < cortex_forward_workspace_bytes(cell == CELL_DAG ? -1 : cell, lin->num_nodes, H))
    return CORTEX_E_WORKSPACE;
  const int cap = max_coresident(inst.fn, kFwdThreads);
  if (cap <= 0) return CORTEX_E_HIP;
  const int cus = num_cus();
  int S, G;
  int64_t q = knob(CORTEX_KNOB_FWD_NODE_GROUPS);
  if (cell == CORTEX_MVRNN) {
    S = 4;
    if (q <= 0) q = (cus > 0 ? cus : 256) / 4;
  } else {
    S = H / inst.J;
    if (q <= 0) q = (S == 1) ? 1 : ((cus > 0 ? cus : 256) / S);
  }
  if (q < 1) q = 1;
  G = (int)(S * q);
  if (G > cap || G > kMaxGrid) return CORTEX_E_TOO_LARGE;
  a.S = S;
  a.Q = (int32_t)q;
  a.sync = (unsigned int *)d_ws;
  a.timeout = barrier_timeout_ticks();
  set_last_grid(1, G);
  return launch_persistent(inst.fn, G, kFwdThreads, a, stream);
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
  return kSyncBytes;
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
