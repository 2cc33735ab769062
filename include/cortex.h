/*
 * cortex.h - C ABI of the MI355X (gfx950) level-synchronous recursive
 * inference library.
 *
 * The library evaluates recursive models (tree RNNs, tree LSTMs, MV-RNN and
 * grid DAG-RNNs) over a batch of trees or DAGs in two steps:
 *
 *   1. cortex_linearize   - data-structure linearization (Sec. 4.2 "Data
 *                           Structure Linearization", numbering scheme of
 *                           Appendix B): node heights, per-level node lists
 *                           (dynamic batching, Sec. 3.1) and child rows.
 *   2. cortex_tree_forward / cortex_dag_forward
 *                         - the lowered loop nest of Sec. 4.1 ("RA Lowering":
 *                           a leaf loop, then a loop over batches of nodes
 *                           whose dependence is carried by the batch loop,
 *                           Appendix A.4), run as ONE persistent kernel with
 *                           the cell weights resident on chip (kernel fusion
 *                           and model persistence, Sec. 7.2 and 7.3).  Levels
 *                           are ordered per datum: each state element is
 *                           also published as a (value, launch tag) pair in
 *                           the workspace and a consumer waits for exactly
 *                           the elements it reads.  TreeRNN at H = 64
 *                           runs the whole batch, or each tree (unrolled
 *                           recursion, Sec. 3.1), in one workgroup with its
 *                           states in LDS and levels ordered by workgroup
 *                           barriers.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named d_* are DEVICE memory owned by the caller.  The library
 *   never allocates or frees memory.  Scratch space comes from the caller's
 *   workspace (d_ws, ws_bytes); it must be zero-filled before its first use
 *   and then passed back unchanged: a call that ends with *d_status == 0
 *   leaves it ready for the next call.  After a call that ends with a
 *   non-zero status, zero the workspace again before reusing it.  Calls that
 *   overlap in time must use distinct workspaces.
 * - The kernels are persistent: every workgroup of a launch must be resident
 *   at once.  A grid of at most one workgroup per compute unit is launched
 *   with a plain launch (it is resident at once on a GPU not shared with
 *   other persistent work); larger grids use the cooperative launch.  No
 *   wait (device-wide barrier or per-datum wait) spins past its limit: it
 *   then writes CORTEX_ST_BARRIER_TIMEOUT, and every other wait ends.
 * - stream is a hipStream_t (NULL = the default stream).  Every call only
 *   enqueues work on it and returns; nothing is synchronised.
 * - The return value reports host-detectable errors (CORTEX_E_*).  When a
 *   call returns an error it has enqueued nothing.
 * - Data-dependent errors are written by the kernels to *d_status (an int32
 *   in device memory, CORTEX_ST_*; the caller sets it to 0 before the first
 *   call and reads it after synchronising).  A kernel that finds *d_status
 *   non-zero on entry writes no outputs, so a failed linearization makes the
 *   following forward a no-op.
 * - Results are deterministic: the same inputs give bitwise identical outputs
 *   on the same GPU.
 *
 * Interface choices beyond the three calls cortex_linearize,
 * cortex_tree_forward and cortex_dag_forward (with their workspace sizes):
 * - cortex_tree_infer / cortex_dag_infer run the whole path of a batch in one
 *   call (one kernel launch where a fused instance fits), and
 *   cortex_tree_infer_noalloc does the same in a library-owned workspace.
 * - Device status 4 reports an inconsistent linearization handed to a
 *   forward.  The arity K is a host check (CORTEX_E_INVAL outside 1..4): the
 *   child format cannot give a node more than K children.  Status 5 reports
 *   an input index outside the input table, status 6 a workspace whose
 *   launch-tag epoch is used up.
 * - cortex_tree_forward takes x_rows, the row count of d_x_table, so input
 *   indices are range-checked on the device, and takes the weights by
 *   pointer (NULL is a host error; a pointer crosses any FFI unchanged).
 * - Cells are int32_t ids (the width of a C enum is up to the compiler),
 *   including the two TreeGRU cells of the refactoring study (Sec. 7.4).
 * - N == 0 is an empty batch, not an error.
 * - stream is a void * holding a hipStream_t, so this header needs no HIP
 *   header.
 * - Launch knobs (cortex_set_knob) select schedules for the ablation
 *   studies; probes measure the MFMA peak and the level-loop floor.
 *
 * Structure format (Sec. 3: a batch of trees or DAGs whose maximum number of
 * children K is declared up front):
 *   d_children[v*K + s] is the node id in child slot s of node v, or -1 when
 *   the slot is empty.  Node ids are 0..N-1.  Any numbering is accepted.  A
 *   node may be the child of several nodes (DAG), a slot may repeat a child.
 */
#ifndef CORTEX_H
#define CORTEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- host return codes ------------------------------------------------ */
#define CORTEX_OK 0
#define CORTEX_E_INVAL (-1)       /* a NULL pointer, a negative size, K or H out of range */
#define CORTEX_E_HIP (-2)         /* a HIP runtime call failed */
#define CORTEX_E_TOO_LARGE (-3)   /* the launch cannot be made co-resident on the GPU */
#define CORTEX_E_WORKSPACE (-4)   /* ws_bytes is smaller than the *_workspace_bytes figure */

/* ---- device status codes (written to *d_status) -------------------------- */
#define CORTEX_ST_OK 0
#define CORTEX_ST_CHILD_RANGE 1      /* a child index outside [-1, N) */
#define CORTEX_ST_CYCLE 2            /* the structure has a cycle (not a DAG) */
#define CORTEX_ST_BARRIER_TIMEOUT 3  /* a barrier or per-datum wait passed its limit */
#define CORTEX_ST_BAD_LINEARIZATION 4 /* forward was handed an inconsistent linearization */
#define CORTEX_ST_INPUT_RANGE 5      /* an input index outside [-1, rows of the input table) */
#define CORTEX_ST_EPOCH_WRAP 6       /* the forward workspace has served 2^32 - 1 launches: zero it */

/* Cells (Sec. 7.1, Table "Models and datasets"). */
#define CORTEX_TREE_RNN 0            /* h = tanh(W [h_l; h_r] + b); leaf h = x */
#define CORTEX_NARY_TREELSTM 1       /* binary N-ary TreeLSTM; leaf (h, c) = (x, 0) */
#define CORTEX_CHILDSUM_TREELSTM 2   /* child-sum TreeLSTM; input x at every node */
#define CORTEX_MVRNN 3               /* MV-RNN; leaf (p, P) = (a, A) */
#define CORTEX_CHILDSUM_TREEGRU 4    /* child-sum TreeGRU: h = z*h~ + (1-z)*h'; input x at every node */
#define CORTEX_SIMPLE_TREEGRU 5      /* SimpleTreeGRU: h = (1-z)*h' (Sec. 7.4 refactoring study) */

/*
 * Linearization (Sec. 4.2, Appendix B).  Every pointer is device memory
 * allocated by the caller with the capacity shown; cortex_linearize fills it.
 *
 * height(v) = 0 for a node without children, else 1 + max height of its
 * children.  Rows are the nodes sorted by (height, node id): level l (the l-th
 * "batch" of dynamic batching) is the contiguous row range
 * [level_offsets[l], level_offsets[l+1]), level 0 holds the leaves, and no row
 * of a level is a child of another row of the same level.  This numbers the
 * leaves first, the reverse of the paper's Appendix B scheme, with the same
 * contiguity and the same one-compare leaf test (row < level_offsets[1]).
 */
typedef struct {
  int32_t num_nodes;       /* N (input) */
  int32_t max_arity;       /* K (input), 1..4 */
  int32_t *num_levels;     /* [1]     L = 1 + max height (0 when N == 0) */
  int32_t *height;         /* [N]     by node id */
  int32_t *level_offsets;  /* [N+1]   capacity; the first L+1 entries are written */
  int32_t *level_nodes;    /* [N]     row -> node id */
  int32_t *node_row;       /* [N]     node id -> row */
  int32_t *child_rows;     /* [N*K]   row r, slot s -> row of that child, or -1 */
} cortex_lin_t;

/* Cell weights, float32, row-major [out, in] (y = W x means y_o = sum_i W[o,i] x_i).
 * Unused members are NULL.
 *   TREE_RNN           W [H, 2H] (columns 0..H-1 act on slot 0, H..2H-1 on slot 1), b [H]
 *   NARY_TREELSTM      U [2, 5, H, H] = (U_l, U_r), gates (i, f_l, f_r, o, u); b [5, H]
 *   CHILDSUM_TREELSTM  W [4, H, H], U [4, H, H], gates (i, f, o, u); b [4, H]
 *   MVRNN              W [H, 2H], W_M [H, 2H]
 *   CHILDSUM_TREEGRU,  W [3, H, H], U [3, H, H], b [3, H], gates (z, r, h):
 *   SIMPLE_TREEGRU       h~ = sum_k h_k, z = s(W_z x + U_z h~ + b_z),
 *                        r_k = s(W_r x + U_r h_k + b_r) per child,
 *                        h' = tanh(W_h x + U_h sum_k r_k*h_k + b_h)
 */
typedef struct {
  const float *W;
  const float *U;
  const float *b;
  const float *W_M;
} cortex_weights_t;

/* ---- linearization -------------------------------------------------------- */

/* Workspace bytes cortex_linearize needs for N nodes of arity K (0 if invalid). */
size_t cortex_linearize_workspace_bytes(int32_t N, int32_t K);

/*
 * Linearize N nodes of maximum arity K (Sec. 4.2).
 *   d_children  [N*K] int32, -1 = empty slot (not modified)
 *   lin         output arrays (see cortex_lin_t); lin->num_nodes must equal N
 *               and lin->max_arity must equal K
 * Kernel-detected errors: CORTEX_ST_CHILD_RANGE, CORTEX_ST_CYCLE,
 * CORTEX_ST_BARRIER_TIMEOUT (outputs are then undefined).
 * N == 0 is an empty batch: it writes num_levels = 0.
 * A batch beyond one workgroup's LDS (above 4,096 nodes; fewer at arity 3
 * and 4) runs on co-resident workgroups of 1,024 threads, each holding at
 * most 8,192 nodes: CORTEX_E_TOO_LARGE when the GPU cannot hold enough of
 * them (one per compute unit at the kernel's register use: 2,097,152 nodes
 * on 256 CUs).  While each workgroup can own one radix tile of 1,024 nodes
 * (up to 524,288 nodes on 256 CUs, two workgroups per unit beyond 262,144)
 * it keeps its nodes' children in registers; larger batches take several
 * height rounds and cost about three times as much per node (655,360
 * nodes: 315 us, against 95 us for 524,288).
 */
int cortex_linearize(const int32_t *d_children, int32_t N, int32_t K, const cortex_lin_t *lin,
                     int32_t *d_status, void *d_ws, size_t ws_bytes, void *stream);

/* ---- forward ------------------------------------------------------------- */

/* Workspace bytes the forward entry points need for a cell (or -1 for the
 * DAG cell) with N nodes and hidden size H (0 if invalid). */
size_t cortex_forward_workspace_bytes(int32_t cell, int32_t N, int32_t H);

/*
 * Forward pass of a tree cell over a linearized batch (the loop nest of
 * Sec. 4.1: a specialized leaf loop, then one fused step per level).
 *   cell        CORTEX_TREE_RNN / NARY_TREELSTM / CHILDSUM_TREELSTM / MVRNN /
 *               CHILDSUM_TREEGRU / SIMPLE_TREEGRU
 *   H           hidden size: 64, 256 or 512 for TREE_RNN, the CHILDSUM TreeLSTM
 *               and the TREEGRU cells; 64 or 256 for NARY; 64 or 128 for MVRNN
 *               (other sizes return CORTEX_E_INVAL and enqueue nothing)
 *   lin         the output of cortex_linearize (K must be 2, or 1..4 for the
 *               child-sum TreeLSTM and TreeGRU cells)
 *   d_x_table   [x_rows, H] float32: leaf vectors or an embedding table
 *   d_x_index   [N] int32 by NODE ID: the input row of each node, -1 = none
 *               (zero input).  TREE_RNN, NARY and MVRNN read it at leaves only;
 *               the child-sum TreeLSTM and TreeGRU cells read it at every node.
 *   d_leaf_mat  MVRNN only: [x_rows, H, H] leaf matrices (row-major)
 *   w           weights (layouts above)
 *   d_h         [N, H] output, in ROW order (row r = node lin->level_nodes[r])
 *   d_c_or_P    NARY/CHILDSUM: [N, H] memory cells; MVRNN: [N, H, H] matrices;
 *               TREE_RNN and the TreeGRU cells: unused (may be NULL).  Row order.
 * An absent child slot contributes a zero state (Sec. 4.3).
 */
int cortex_tree_forward(int32_t cell, int32_t H, const cortex_lin_t *lin, const float *d_x_table,
                        int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                        const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status,
                        void *d_ws, size_t ws_bytes, void *stream);

/*
 * The whole hot path of a tree batch in one call: the linearization of
 * cortex_linearize (written to *lin) followed by cortex_tree_forward, with the
 * arguments and results of those two calls (N and K are taken from lin).
 * Where the cell has a fused instance -- TreeRNN (H = 64 up to 320 nodes,
 * 256, 512), N-ary TreeLSTM (64, 256), child-sum TreeLSTM and the TreeGRU
 * cells (64, 256, 512), MV-RNN (d = 64); N <= 2048, the schedule knobs at their defaults
 * (FWD_NODE_GROUPS aside) and the batch's linearization and structure
 * fitting one compute unit's LDS beside the kernel's own -- this is ONE
 * kernel launch: every workgroup linearizes the batch in LDS for itself (the
 * single-workgroup linearizer's algorithm) and workgroup 0 writes *lin out.
 * Otherwise (MV-RNN at d = 128, larger batches) it enqueues cortex_linearize,
 * then cortex_tree_forward.
 *   d_children  [N*K] int32 by node id, -1 = absent slot (as cortex_linearize)
 *   d_ws        cortex_tree_infer_workspace_bytes(cell, N, K, H) bytes of
 *               device memory, zeroed before its first use (the linearizer's
 *               workspace, then the forward's)
 * Host errors return CORTEX_E_* and enqueue nothing; a child index out of
 * range, a cycle or a broken input index set *d_status as the two calls do.
 */
size_t cortex_tree_infer_workspace_bytes(int32_t cell, int32_t N, int32_t K, int32_t H);
int cortex_tree_infer(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                      const float *d_x_table, int32_t x_rows, const int32_t *d_x_index, const float *d_leaf_mat,
                      const cortex_weights_t *w, float *d_h, float *d_c_or_P, int32_t *d_status, void *d_ws,
                      size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * cortex_tree_infer with the workspace taken from a library-owned array in
 * device memory instead of a caller's buffer.  The caller still passes the
 * linearization arrays, inputs, weights, outputs and status word, with the
 * meanings of cortex_tree_infer; the results are bitwise those of
 * cortex_tree_infer on the same inputs.
 *   - The array is CORTEX_NOALLOC_SCRATCH_BYTES per GPU, held from the first
 *     call on that GPU until the process ends.  The call allocates nothing:
 *     no hipMalloc, no hipFree, no allocating library routine.
 *   - Size limits (each checked on the host): the linearizer workspace
 *     (cortex_linearize_workspace_bytes, needed when the batch takes two
 *     launches) at most 2 MiB; N * H at most 2,097,152 for the h staging;
 *     the second state's staging (c and the TreeGRU reset sums: N * H; P of
 *     MV-RNN: N * H * H) at most 4,194,304 elements; the TreeGRU phase values
 *     (N * H * 3 floats) at most 8 MiB.  A batch beyond them returns
 *     CORTEX_E_WORKSPACE and enqueues nothing.  Other host errors are those of
 *     cortex_tree_infer, also with nothing enqueued.
 *   - Each call enqueues, before the path's own launches, one small kernel
 *     that prepares the array (it clears its barrier words and advances its
 *     staging epoch; the first call on a GPU clears the whole array).  So a
 *     call after one that ended with a non-zero status needs no reset beyond
 *     setting *d_status back to 0.
 *   - Every call on a GPU shares that GPU's array, which keeps the last
 *     call's contents: calls that overlap in time on one GPU (other streams,
 *     other threads) race and give wrong results.  Order them, e.g. on one
 *     stream.
 */
#define CORTEX_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
int cortex_tree_infer_noalloc(int32_t cell, int32_t H, const int32_t *d_children, const cortex_lin_t *lin,
                              const float *d_x_table, int32_t x_rows, const int32_t *d_x_index,
                              const float *d_leaf_mat, const cortex_weights_t *w, float *d_h, float *d_c_or_P,
                              int32_t *d_status, void *stream);

/*
 * Forward pass of the DAG-RNN cell (recursive part of DAG-RNN, Sec. 7.1):
 *   h(v) = tanh(W x(v) + U_0 h(slot 0) + U_1 h(slot 1) + b)
 * (for image grids slot 0 is the node above, slot 1 the node to the left).
 *   H      64, 256 or 512
 *   lin    the output of cortex_linearize with K == 2
 *   d_x    [N, H] float32 input by NODE ID
 *   d_W    [H, H];  d_U [2, H, H] (slot 0 then slot 1);  d_b [H]
 *   d_h    [N, H] output in ROW order
 * Every node, sources included, runs the cell; an empty slot contributes 0.
 */
int cortex_dag_forward(int32_t H, const cortex_lin_t *lin, const float *d_x, const float *d_W,
                       const float *d_U, const float *d_b, float *d_h, int32_t *d_status,
                       void *d_ws, size_t ws_bytes, void *stream);

/*
 * The whole hot path of a DAG-RNN batch in one call: cortex_linearize, then
 * cortex_dag_forward, with the arguments and results of those two calls.  One
 * kernel launch where the batch fits the fused instance of the kernel with
 * 16-unit slices (H = 64 or 512, or 256 below the 64-unit kernel's range of
 * 6144 nodes; N <= 2048, default schedule knobs, the linearization fitting
 * one compute unit's LDS beside the weight slice): every workgroup linearizes
 * the batch in LDS and workgroup 0 writes *lin out.  Otherwise the two calls.
 *   d_ws   cortex_dag_infer_workspace_bytes(N, K, H) bytes, zeroed before first use
 */
size_t cortex_dag_infer_workspace_bytes(int32_t N, int32_t K, int32_t H);
int cortex_dag_infer(int32_t H, const int32_t *d_children, const cortex_lin_t *lin, const float *d_x,
                     const float *d_W, const float *d_U, const float *d_b, float *d_h, int32_t *d_status,
                     void *d_ws, size_t ws_bytes, void *stream);

/* ---- tuning and diagnostics ---------------------------------------------- */

/*
 * Launch knobs, process-wide, read at each launch.  They change the schedule,
 * not what is computed: outputs are bitwise those of the defaults, except where
 * a knob picks a kernel that adds partial sums in another order (DAG-RNN slice
 * width, TREE_UNROLL = 1), whose states agree to rounding.
 *   CORTEX_KNOB_LIN_BLOCKS          workgroups of the linearizer (0 = chosen from N)
 *   CORTEX_KNOB_FWD_NODE_GROUPS     node groups of the forward; workgroups =
 *                                   hidden slices x node groups (0 = fill the
 *                                   GPU; a kernel with one slice, TreeRNN at
 *                                   H = 64, takes one group per 16 nodes, at
 *                                   most one per compute unit)
 *   CORTEX_KNOB_BARRIER_TIMEOUT_US  spin limit of one barrier or per-datum wait in
 *                                   microseconds (default 200,000: 0.2 s; 0 makes every
 *                                   wait time out at once, for tests of that path)
 *   CORTEX_KNOB_COOPERATIVE         1 = always use the cooperative launch
 *                                   (0 = only when the grid exceeds one
 *                                   workgroup per compute unit)
 *   CORTEX_KNOB_FWD_SLICE_UNITS     hidden units per workgroup slice of the
 *                                   forward (0 = the default of the cell;
 *                                   other values are used where the library
 *                                   has a kernel for them: 2 for the N-ary
 *                                   TreeLSTM at H = 256; 16 or 64 for the
 *                                   DAG-RNN at H = 256, whose default is 64
 *                                   for batches of at least 6144 nodes and
 *                                   16 below)
 *   CORTEX_KNOB_LEVEL_SYNC          how the forward orders its levels, for
 *                                   ablation studies (the results are the same):
 *                                   0 = per-datum waits in one launch (default);
 *                                   1 = also a device-wide barrier after every
 *                                   level (slice and child-sum kernels);
 *                                   2 = one launch per level, each reloading
 *                                   weights and structure (slice, child-sum
 *                                   and 64-unit DAG-RNN kernels; the call then
 *                                   synchronizes the stream once to read L);
 *                                   3 = the TreeGRU cells only: a device-wide
 *                                   barrier after each of a level's two
 *                                   exchanges (the reset sums, then the
 *                                   states): the TreeGRU schedule without
 *                                   recursive refactoring (Secs. 3.1, 7.4), where
 *                                   1 is the refactored one.
 *                                   A forward whose kernel lacks the mode
 *                                   returns CORTEX_E_INVAL.
 *   CORTEX_KNOB_TREE_UNROLL         TreeRNN at H = 64 (Secs. 3.1, 7.4, unrolled
 *                                   recursion): 0 = the default choice (the
 *                                   whole batch in one workgroup up to 320
 *                                   nodes, one workgroup per tree up to 2048,
 *                                   hidden slices beyond); 1 = level-parallel
 *                                   hidden slices, states exchanged between
 *                                   workgroups at every level; 2 = one
 *                                   workgroup per tree, each tree evaluated
 *                                   leaves to root on one compute unit (up to
 *                                   2048 nodes, else CORTEX_E_INVAL; with
 *                                   FWD_NODE_GROUPS > 0 that many workgroups
 *                                   share the trees).
 *   CORTEX_KNOB_ABLATE              bit mask switching optimizations off, for
 *                                   ablation studies (Sec. 7.3; the results are
 *                                   the same): bit 0 = no model persistence,
 *                                   the weight slice is read from the weight
 *                                   tensors at every tile instead of staying
 *                                   in LDS; bit 1 = no leaf specialization,
 *                                   leaf states are staged and their parents
 *                                   wait for them instead of reading the
 *                                   inputs directly.  Slice kernels only
 *                                   (TreeRNN at H = 256 / 512, N-ary TreeLSTM;
 *                                   bit 0 also DAG-RNN with 16-unit slices).
 *                                   Bit 2 = input products hoisted (Sec. 7.1):
 *                                   W x + b of every node is computed by one
 *                                   matrix-product launch before the level
 *                                   loop (into d_h, which the loop then
 *                                   overwrites) instead of inside each tile;
 *                                   DAG-RNN with 64-unit slices only, results
 *                                   equal to rounding.  Other forwards return
 *                                   CORTEX_E_INVAL.
 * cortex_set_knob returns CORTEX_E_INVAL for an unknown knob or a negative value
 * (or a LEVEL_SYNC value above 3, an ABLATE value above 7, a TREE_UNROLL
 * value above 2).
 */
#define CORTEX_KNOB_LIN_BLOCKS 0
#define CORTEX_KNOB_FWD_NODE_GROUPS 1
#define CORTEX_KNOB_BARRIER_TIMEOUT_US 2
#define CORTEX_KNOB_COOPERATIVE 3
#define CORTEX_KNOB_FWD_SLICE_UNITS 4
#define CORTEX_KNOB_LEVEL_SYNC 5
#define CORTEX_KNOB_TREE_UNROLL 6
#define CORTEX_KNOB_ABLATE 7
int cortex_set_knob(int32_t knob, int64_t value);
int64_t cortex_get_knob(int32_t knob);

/* Workgroups the last launch of each kind used (for reports; host-side). */
int32_t cortex_last_grid(int32_t which /* 0 = linearize, 1 = forward */);

/* Matrix-core throughput probe, for reporting achieved rates beside a sustained
 * (measured) peak as well as the nominal one.  cortex_probe_mfma enqueues one
 * workgroup of 8 waves per compute unit on `stream`; every wave runs `iters`
 * rounds of 16 chained v_mfma_f32_16x16x4_f32 on register operands (no memory
 * traffic) and writes one float per lane to d_sink, which must hold
 * cortex_probe_mfma_sink_floats() floats (device memory, caller-owned).
 * cortex_probe_mfma_flops(iters) is the fp32 flop count of one such launch
 * (2 x 16 x 16 x 4 per instruction).  Returns CORTEX_E_INVAL for a NULL sink or
 * negative iters, CORTEX_E_HIP if the device cannot be queried or the launch
 * fails; the sizes return 0 then.  The sink values carry no meaning. */
size_t cortex_probe_mfma_sink_floats(void);
double cortex_probe_mfma_flops(int32_t iters);
int cortex_probe_mfma(float *d_sink, int32_t iters, void *stream);

/* Level-ordering probe, for the fixed cost a level loop pays before any work:
 * a persistent launch of `grid` workgroups of 512 threads (1 <= grid <= the
 * number of compute units, one per unit, as the forward kernels launch) that
 * runs `levels` empty levels.  mode 0 ends each level with a device-wide
 * barrier; mode 1 orders levels per datum as the forward kernels do: every
 * workgroup publishes one (value, tag) pair, in a 128-byte line of its own,
 * with a device-scope store and waits until the pair of every workgroup
 * carries that level's tag.
 * levels = 0 measures the launch alone.  d_ws (device, caller-owned, at least
 * cortex_probe_levels_workspace_bytes()) must be zeroed before its first use
 * and again after a launch that ended with a non-zero *d_status; every wait is
 * bounded by CORTEX_KNOB_BARRIER_TIMEOUT_US and raises
 * CORTEX_ST_BARRIER_TIMEOUT when it runs out.  Returns CORTEX_E_INVAL (NULL
 * pointer, mode not 0 or 1, levels < 0, grid < 1), CORTEX_E_TOO_LARGE (grid
 * above the compute-unit count), CORTEX_E_WORKSPACE or CORTEX_E_HIP, and then
 * enqueues nothing.  Calls that share a workspace must not overlap. */
size_t cortex_probe_levels_workspace_bytes(void);
int cortex_probe_levels(int32_t mode, int32_t grid, int32_t levels, int32_t *d_status, void *d_ws,
                        size_t ws_bytes, void *stream);

/* Library version string. */
const char *cortex_version(void);

#ifdef __cplusplus
}
#endif
#endif /* CORTEX_H */
