"""Seeded synthetic workloads for level-synchronous recursive inference.

This module only draws random structures and tensors.  It holds none of the
method's arithmetic (no heights, no levels, no cell evaluation): both the HIP
path and the fp64 oracle consume the arrays it returns, so it is the one piece
of code the two sides share.

Structure format (the paper's problem statement, Sec. 3 "Recursive API": a
batch of trees or DAGs with a declared maximum number of children):

* ``children``: int32 ``[N*K]``, row-major by node id; slot ``s`` of node ``v``
  is ``children[v*K+s]`` and ``-1`` marks an absent slot.
* Trees are numbered in post-order, tree after tree, child slots in creation
  order.  Grid DAGs are numbered ``g*R*C + i*C + j`` with slot 0 the node above
  ``(i-1, j)`` and slot 1 the node to the left ``(i, j-1)``.

Float data are drawn in float64 and cast once to float32; both sides read the
float32 arrays.  Draw order within a workload: structure (sizes first, then
splits or arities), then input ids, then input tables and leaf data, then the
weight matrices in the order listed, then the biases.

The five named workloads stand in for the paper's evaluation models (Table
"Models and datasets", Sec. 7.1): TreeFC/TreeRNN, binary and child-sum
TreeLSTM, MV-RNN and the recursive part of DAG-RNN.  The Stanford Sentiment Treebank is
not available, so SST-sized random trees (10-40 leaves, batch 10) replace it.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

BASE_SEED = 13830

CELL_TREE_RNN = "tree_rnn"
CELL_NARY_TREELSTM = "nary_treelstm"
CELL_CHILDSUM_TREELSTM = "childsum_treelstm"
CELL_MVRNN = "mvrnn"
CELL_DAGRNN = "dagrnn"
CELL_CHILDSUM_TREEGRU = "childsum_treegru"
CELL_SIMPLE_TREEGRU = "simple_treegru"


@dataclass
class Workload:
    """One batch of structures plus the inputs and weights of one cell."""

    name: str
    cell: str
    H: int
    K: int
    children: np.ndarray                      # int32 [N*K]
    x_index: Optional[np.ndarray] = None      # int32 [N], -1 = no input
    x_table: Optional[np.ndarray] = None      # float32 [V, H] (leaf vectors / embeddings)
    leaf_mat: Optional[np.ndarray] = None     # float32 [V, H, H] (MV-RNN leaf matrices)
    x: Optional[np.ndarray] = None            # float32 [N, H] (DAG-RNN per-node input)
    W: Optional[np.ndarray] = None
    U: Optional[np.ndarray] = None
    b: Optional[np.ndarray] = None
    W_M: Optional[np.ndarray] = None
    meta: Dict[str, object] = field(default_factory=dict)

    @property
    def N(self) -> int:
        return int(self.children.size // self.K)


# ---------------------------------------------------------------------------
# Tree shapes
# ---------------------------------------------------------------------------

def random_split_tree(rng: np.random.Generator, n_leaves: int) -> list:
    """Binary tree with ``n_leaves`` leaves by recursive random splits.

    split(n): one leaf if n == 1, else draw k ~ U{1..n-1} and build
    split(k) as the left subtree and split(n-k) as the right one.  The draw is
    made before recursing (pre-order).  A tree is a nested list: ``[]`` is a
    leaf, ``[left, right]`` an internal node.
    """
    if n_leaves < 1:
        raise ValueError("a tree needs at least one leaf")
    # explicit stack so that deep (caterpillar-like) splits cannot hit Python's
    # recursion limit; the visiting order equals the recursive pre-order
    root: list = []
    stack: List[Tuple[list, int]] = [(root, n_leaves)]
    while stack:
        node, n = stack.pop()
        if n == 1:
            continue
        k = int(rng.integers(1, n))
        left: list = []
        right: list = []
        node.extend([left, right])
        stack.append((right, n - k))
        stack.append((left, k))
    return root


def random_arity_tree(rng: np.random.Generator, n_nodes: int, max_arity: int = 4) -> list:
    """Tree with ``n_nodes`` nodes grown breadth-first with random arity.

    Pop the oldest open node, draw a ~ U{1..max_arity} and give it
    min(a, n_nodes - created) new children; stop once ``n_nodes`` exist.  The
    nodes still open are leaves.
    """
    if n_nodes < 1:
        raise ValueError("a tree needs at least one node")
    root: list = []
    created = 1
    queue = [root]
    head = 0
    while created < n_nodes and head < len(queue):
        node = queue[head]
        head += 1
        a = int(rng.integers(1, max_arity + 1))
        for _ in range(min(a, n_nodes - created)):
            kid: list = []
            node.append(kid)
            queue.append(kid)
            created += 1
    return root


def perfect_tree(height: int) -> list:
    """Perfect binary tree; ``height`` counts edges (height 0 is one leaf)."""
    if height == 0:
        return []
    return [perfect_tree(height - 1), perfect_tree(height - 1)]


def caterpillar(n_leaves: int, left_spine: bool = True) -> list:
    """Chain-shaped binary tree: every internal node has one leaf child.

    ``left_spine=True`` puts the spine in slot 0 (the previous internal node
    on the left, a fresh leaf on the right).
    """
    t: list = []
    for _ in range(n_leaves - 1):
        t = [t, []] if left_spine else [[], t]
    return t


def forest_to_children(trees: List[list], K: int) -> Tuple[np.ndarray, np.ndarray]:
    """Post-order numbering of a forest, tree after tree.

    Returns ``(children[N*K] int32, is_leaf[N] bool)``.
    """
    kids_of: List[List[int]] = []

    for t in trees:
        # iterative post-order: children (left to right) before the parent
        stack: List[Tuple[list, int, List[int]]] = [(t, 0, [])]
        while stack:
            node, nxt, got = stack[-1]
            if nxt < len(node):
                stack[-1] = (node, nxt + 1, got)
                stack.append((node[nxt], 0, []))
                continue
            stack.pop()
            if len(got) > K:
                raise ValueError(f"node has {len(got)} children > K={K}")
            vid = len(kids_of)
            kids_of.append(list(got))
            if stack:
                stack[-1][2].append(vid)
    N = len(kids_of)
    children = np.full(N * K, -1, dtype=np.int32)
    for v, ks in enumerate(kids_of):
        children[v * K: v * K + len(ks)] = ks
    is_leaf = np.array([len(ks) == 0 for ks in kids_of], dtype=bool)
    return children, is_leaf


def grid_children(n_grids: int, rows: int, cols: int) -> np.ndarray:
    """Grid DAGs: node (g,i,j) reads (i-1,j) in slot 0 and (i,j-1) in slot 1."""
    N = n_grids * rows * cols
    children = np.full(N * 2, -1, dtype=np.int32)
    for g in range(n_grids):
        base = g * rows * cols
        for i in range(rows):
            for j in range(cols):
                v = base + i * cols + j
                if i > 0:
                    children[2 * v] = base + (i - 1) * cols + j
                if j > 0:
                    children[2 * v + 1] = base + i * cols + (j - 1)
    return children


def _u(rng, lo, hi, shape):
    return rng.uniform(lo, hi, size=shape).astype(np.float32)


def _n(rng, shape, std=1.0):
    return (rng.standard_normal(size=shape) * std).astype(np.float32)


# ---------------------------------------------------------------------------
# Named workloads
# ---------------------------------------------------------------------------

def tree_rnn_workload(seed: int, n_leaves: int = 32, H: int = 64) -> Workload:
    """One binary tree of ``n_leaves`` leaves; h = tanh(W[h_l;h_r] + b), b = 0."""
    rng = np.random.default_rng(seed)
    tree = random_split_tree(rng, n_leaves)
    children, is_leaf = forest_to_children([tree], 2)
    N = is_leaf.size
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = np.arange(int(is_leaf.sum()), dtype=np.int32)
    leaves = _n(rng, (int(is_leaf.sum()), H))
    W = _u(rng, -0.1, 0.1, (H, 2 * H))
    b = np.zeros(H, dtype=np.float32)
    return Workload("tree_rnn_h%d_1x%d" % (H, n_leaves), CELL_TREE_RNN, H, 2, children,
                    x_index=x_index, x_table=leaves, W=W, b=b)


def tree_rnn_forest_workload(seed: int, batch: int = 10, H: int = 64, leaf_lo: int = 32, leaf_hi: int = 32,
                             shuffle: bool = False) -> Workload:
    """A batch of TreeRNN trees (random splits, leaf counts drawn from
    [leaf_lo, leaf_hi]); the cell and weight recipe of the one-tree workload.
    ``shuffle`` renames the nodes by a random permutation, so the trees of the
    batch interleave in id order."""
    rng = np.random.default_rng(seed)
    children, is_leaf = _binary_forest(rng, batch, leaf_lo, leaf_hi)
    N = is_leaf.size
    if shuffle:
        perm = rng.permutation(N).astype(np.int32)
        children = relabel(children, 2, perm)
        moved = np.zeros(N, dtype=bool)
        moved[perm] = is_leaf
        is_leaf = moved
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = np.arange(int(is_leaf.sum()), dtype=np.int32)
    leaves = _n(rng, (int(is_leaf.sum()), H))
    W = _u(rng, -0.1, 0.1, (H, 2 * H))
    b = np.zeros(H, dtype=np.float32)
    name = "tree_rnn_h%d_%dx%d" % (H, batch, leaf_lo) if leaf_lo == leaf_hi else \
        "tree_rnn_h%d_%dx%d-%d" % (H, batch, leaf_lo, leaf_hi)
    return Workload(name, CELL_TREE_RNN, H, 2, children, x_index=x_index, x_table=leaves, W=W, b=b)


def _binary_forest(rng, batch, leaf_lo, leaf_hi):
    sizes = [int(rng.integers(leaf_lo, leaf_hi + 1)) for _ in range(batch)]
    trees = [random_split_tree(rng, s) for s in sizes]
    return forest_to_children(trees, 2)


def nary_treelstm_workload(seed: int, batch: int = 10, H: int = 256, vocab: int = 1000,
                           leaf_lo: int = 10, leaf_hi: int = 40) -> Workload:
    """Binary N-ary TreeLSTM: leaves read Emb[id]; gates (i, f_l, f_r, o, u)."""
    rng = np.random.default_rng(seed)
    children, is_leaf = _binary_forest(rng, batch, leaf_lo, leaf_hi)
    N = is_leaf.size
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = rng.integers(0, vocab, size=int(is_leaf.sum())).astype(np.int32)
    emb = _n(rng, (vocab, H))
    U = np.stack([_u(rng, -0.05, 0.05, (5, H, H)), _u(rng, -0.05, 0.05, (5, H, H))])
    b = _u(rng, -0.05, 0.05, (5, H))
    return Workload("nary_treelstm_h%d_b%d" % (H, batch), CELL_NARY_TREELSTM, H, 2, children,
                    x_index=x_index, x_table=emb, U=U, b=b)


def childsum_treelstm_workload(seed: int, batch: int = 10, H: int = 256, vocab: int = 1000,
                               node_lo: int = 20, node_hi: int = 80, max_arity: int = 4) -> Workload:
    """Child-sum TreeLSTM over random-arity trees; every node reads Emb[id]."""
    rng = np.random.default_rng(seed)
    sizes = [int(rng.integers(node_lo, node_hi + 1)) for _ in range(batch)]
    trees = [random_arity_tree(rng, s, max_arity) for s in sizes]
    children, is_leaf = forest_to_children(trees, max_arity)
    N = is_leaf.size
    x_index = rng.integers(0, vocab, size=N).astype(np.int32)
    emb = _n(rng, (vocab, H))
    W = _u(rng, -0.05, 0.05, (4, H, H))
    U = _u(rng, -0.05, 0.05, (4, H, H))
    b = _u(rng, -0.05, 0.05, (4, H))
    return Workload("childsum_treelstm_h%d_b%d" % (H, batch), CELL_CHILDSUM_TREELSTM, H,
                    max_arity, children, x_index=x_index, x_table=emb, W=W, U=U, b=b)


def childsum_treegru_workload(seed: int, batch: int = 10, H: int = 256, vocab: int = 1000,
                              node_lo: int = 20, node_hi: int = 80, max_arity: int = 4,
                              simple: bool = False) -> Workload:
    """Child-sum TreeGRU (or SimpleTreeGRU) over random-arity trees, the same
    shapes as the child-sum TreeLSTM; every node reads Emb[id]; weights
    W, U [3, H, H] and b [3, H] (gates z, r, h) ~ U(-0.05, 0.05)."""
    rng = np.random.default_rng(seed)
    sizes = [int(rng.integers(node_lo, node_hi + 1)) for _ in range(batch)]
    trees = [random_arity_tree(rng, s, max_arity) for s in sizes]
    children, is_leaf = forest_to_children(trees, max_arity)
    N = is_leaf.size
    x_index = rng.integers(0, vocab, size=N).astype(np.int32)
    emb = _n(rng, (vocab, H))
    W = _u(rng, -0.05, 0.05, (3, H, H))
    U = _u(rng, -0.05, 0.05, (3, H, H))
    b = _u(rng, -0.05, 0.05, (3, H))
    cell = CELL_SIMPLE_TREEGRU if simple else CELL_CHILDSUM_TREEGRU
    name = ("simple_treegru_h%d_b%d" if simple else "childsum_treegru_h%d_b%d") % (H, batch)
    return Workload(name, cell, H, max_arity, children, x_index=x_index, x_table=emb, W=W, U=U, b=b)


def mvrnn_workload(seed: int, batch: int = 10, d: int = 64, leaf_lo: int = 10,
                   leaf_hi: int = 40, wm_scale: float = 0.1) -> Workload:
    """MV-RNN: leaf (a, A) = (N(0,1), I + 0.01 N(0,1)); p = tanh(W[Ba; Ab]), P = W_M[A; B]."""
    rng = np.random.default_rng(seed)
    children, is_leaf = _binary_forest(rng, batch, leaf_lo, leaf_hi)
    N = is_leaf.size
    n_leaf = int(is_leaf.sum())
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = np.arange(n_leaf, dtype=np.int32)
    a = _n(rng, (n_leaf, d))
    A = (np.eye(d)[None, :, :] + 0.01 * rng.standard_normal(size=(n_leaf, d, d))).astype(np.float32)
    W = _u(rng, -0.1, 0.1, (d, 2 * d))
    W_M = _u(rng, -wm_scale, wm_scale, (d, 2 * d))
    return Workload("mvrnn_d%d_b%d" % (d, batch), CELL_MVRNN, d, 2, children,
                    x_index=x_index, x_table=a, leaf_mat=A, W=W, W_M=W_M)


def dagrnn_workload(seed: int, n_grids: int = 64, rows: int = 32, cols: int = 32,
                    H: int = 256) -> Workload:
    """Grid DAG-RNN: h(i,j) = tanh(W x + U_up h(i-1,j) + U_left h(i,j-1) + b)."""
    rng = np.random.default_rng(seed)
    children = grid_children(n_grids, rows, cols)
    N = n_grids * rows * cols
    x = _n(rng, (N, H))
    W = _u(rng, -0.05, 0.05, (H, H))
    U = np.stack([_u(rng, -0.05, 0.05, (H, H)), _u(rng, -0.05, 0.05, (H, H))])
    b = _u(rng, -0.05, 0.05, (H,))
    return Workload("dagrnn_h%d_%dx%dx%d" % (H, n_grids, rows, cols), CELL_DAGRNN, H, 2,
                    children, x=x, W=W, U=U, b=b)


def treefc_workload(seed: int, batch: int = 10, height: int = 7, H: int = 256) -> Workload:
    """TreeFC (the paper's TF-Fold benchmarking model, Table "Models and
    datasets"): ``batch`` perfect binary trees of height ``height`` (edges),
    read as the TreeRNN cell h = tanh(W[h_l; h_r] + b) with leaf h = N(0,1)
    rows; W, b ~ U(-0.05, 0.05)."""
    rng = np.random.default_rng(seed)
    children, is_leaf = forest_to_children([perfect_tree(height) for _ in range(batch)], 2)
    N = is_leaf.size
    n_leaf = int(is_leaf.sum())
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = np.arange(n_leaf, dtype=np.int32)
    leaves = _n(rng, (n_leaf, H))
    W = _u(rng, -0.05, 0.05, (H, 2 * H))
    b = _u(rng, -0.05, 0.05, (H,))
    return Workload("treefc_h%d_b%d" % (H, batch), CELL_TREE_RNN, H, 2, children,
                    x_index=x_index, x_table=leaves, W=W, b=b)


# The paper's evaluation grid (Sec. 7.1, Table "Models and datasets"; its
# latency table lists batch sizes 1 and 10 and hidden sizes h_s / h_l =
# 256 / 512, 64 / 128 for MV-RNN).  SST-based models (TreeGRU, TreeLSTM,
# MV-RNN) use the SST-sized random trees of the five workloads above.
PAPER_GRID_CELLS = ("treefc", "dagrnn", "treegru", "treelstm", "mvrnn")


def paper_grid_workload(cell: str, batch: int, hidden: str) -> Workload:
    """One cell of the paper's grid; ``hidden`` is "s" or "l"."""
    idx = PAPER_GRID_CELLS.index(cell) * 4 + (0 if batch == 1 else 1) * 2 + (0 if hidden == "s" else 1)
    seed = BASE_SEED + 1000 + idx
    if cell == "treefc":
        return treefc_workload(seed, batch=batch, H=256 if hidden == "s" else 512)
    if cell == "dagrnn":
        return dagrnn_workload(seed, n_grids=batch, rows=10, cols=10, H=256 if hidden == "s" else 512)
    if cell == "treelstm":
        return childsum_treelstm_workload(seed, batch=batch, H=256 if hidden == "s" else 512)
    if cell == "treegru":
        return childsum_treegru_workload(seed, batch=batch, H=256 if hidden == "s" else 512)
    if cell == "mvrnn":
        return mvrnn_workload(seed, batch=batch, d=64 if hidden == "s" else 128)
    raise ValueError(cell)


# The five evaluation workloads, indexed 0..4.  Extra parity seeds for workload
# k are BASE_SEED + 100*j + k + 1 (j = 1, 2, ...).
WORKLOADS = {
    0: ("tree_rnn_h64_1x32", tree_rnn_workload),
    1: ("nary_treelstm_h256_b10", nary_treelstm_workload),
    2: ("childsum_treelstm_h256_b10", childsum_treelstm_workload),
    3: ("mvrnn_d64_b10", mvrnn_workload),
    4: ("dagrnn_h256_64x32x32", dagrnn_workload),
}


def workload_seed(k: int, j: int = 0) -> int:
    return BASE_SEED + 100 * j + k + 1


def make_workload(k: int, j: int = 0, **kw) -> Workload:
    """Workload ``k`` (0..4) at seed variant ``j`` (0 = the canonical seed)."""
    _, fn = WORKLOADS[k]
    return fn(workload_seed(k, j), **kw)


def relabel(children: np.ndarray, K: int, perm: np.ndarray) -> np.ndarray:
    """Rename node v to perm[v] (a permutation); slot order is kept."""
    N = children.size // K
    out = np.full(N * K, -1, dtype=np.int32)
    ch = children.reshape(N, K)
    for v in range(N):
        for s in range(K):
            c = ch[v, s]
            out[perm[v] * K + s] = -1 if c < 0 else perm[c]
    return out


def random_dag(rng: np.random.Generator, N: int, K: int, p_absent: float = 0.3) -> np.ndarray:
    """Random DAG over ids 0..N-1: each slot of v points to a random lower id
    (or is absent), then ids are shuffled so the order carries no hint."""
    ch = np.full((N, K), -1, dtype=np.int32)
    for v in range(1, N):
        for s in range(K):
            if rng.random() >= p_absent:
                ch[v, s] = int(rng.integers(0, v))
    perm = rng.permutation(N).astype(np.int32)
    return relabel(ch.reshape(-1), K, perm)
