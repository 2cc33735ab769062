"""fp64 CPU oracle for level-synchronous recursive inference.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no
code with the HIP library and the HIP library never calls it.

What it computes
----------------
Properties P.1-P.3 (Sec. 2 "Overview") say that control flow depends only on
the structure, that every recursive call can be made before any tensor work,
and that sibling calls are independent.  Hence any order that evaluates
children before parents gives the same per-node result, and level batching
(dynamic batching, Sec. 3.1; lowering to loops, Sec. 4.1) is one such order.
The oracle is therefore the plain recursive definition:

* ``linearize``: node heights by recursion, rows by sorting on (height, id),
  level offsets by counting, child rows by lookup (Sec. 4.2 "Data Structure
  Linearization"; numbering scheme of Appendix B, with the reading that rows
  ascend from the leaves).
* ``forward``: a memoized recursive evaluator (the running example of Sec. 3,
  leaf case + recursive case) returning every node's state in node-id order.
* ``forward_levels``: the same cell evaluated level by level over the
  linearization (the loop nest of Sec. 4.1), used to check order invariance.
* ``dfs_batches``: the depth-first, post-order batching the paper describes
  for trees (Sec. 4.2), with K slots, used to pin ``linearize``.

All arithmetic is float64 on float32 inputs (upcast once), with
sigma(z) = 1/(1+exp(-z)) and numpy's tanh/exp.  An absent child slot (-1)
contributes a zero state (zero-initial-value hoisting, Sec. 4.3).

Cells (the paper cites but does not print their equations; the standard
published forms are used, see the readings listed with the design notes):

* tree_rnn           h = tanh(W[:, :H] h_l + W[:, H:] h_r + b); leaf h = x
* nary_treelstm      gates (i, f_l, f_r, o, u) from U_l h_l + U_r h_r + b;
                     c = i*u + f_l*c_l + f_r*c_r, h = o*tanh(c); leaf (x, 0)
* childsum_treelstm  h~ = sum_k h_k; i, o, u from W x + U h~ + b, one forget
                     gate per child from W_f x + U_f h_k + b_f;
                     c = i*u + sum_k f_k*c_k, h = o*tanh(c); x at every node
* mvrnn              p = tanh(W [B a; A b]), P = W_M [A; B]; leaf (a, A)
* dagrnn             h = tanh(W x + U_up h_up + U_left h_left + b)
* childsum_treegru   h~ = sum_k h_k; z = sig(W_z x + U_z h~ + b_z); one reset
                     gate per child r_k = sig(W_r x + U_r h_k + b_r);
                     h' = tanh(W_h x + U_h sum_k r_k*h_k + b_h);
                     h = z*h~ + (1-z)*h'; x at every node
* simple_treegru     the same with h = (1-z)*h' (the simplification the
                     paper describes for its refactoring study, Sec. 7.4)

Every function here is pinned by ``tests/test_oracle_*.py`` against hand
values, library cells (torch RNNCell/LSTMCell in fp64), closed forms and the
paper's own linearizer.
"""
from __future__ import annotations

import sys
from contextlib import contextmanager
from typing import Dict, List, Optional, Sequence

import numpy as np


class StructureError(ValueError):
    """Invalid structure: a child index out of range or a cycle."""


class ChildRangeError(StructureError):
    pass


class CycleError(StructureError):
    pass


@contextmanager
def _deep_recursion(depth: int):
    old = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old, depth))
    try:
        yield
    finally:
        sys.setrecursionlimit(old)


def _kids(children: np.ndarray, K: int, v: int) -> List[int]:
    return [int(c) for c in children[v * K:(v + 1) * K]]


# ---------------------------------------------------------------------------
# Linearization (Sec. 4.2; numbering of Appendix B)
# ---------------------------------------------------------------------------

def heights(children: np.ndarray, K: int) -> np.ndarray:
    """height(v) = 0 without children, else 1 + max over present children.

    Raises ChildRangeError for an index outside [-1, N) and CycleError for a
    cycle (a DAG is required by the recursion being well founded).
    """
    children = np.asarray(children, dtype=np.int64)
    N = children.size // K
    if children.size != N * K:
        raise ValueError("children length is not a multiple of K")
    bad = (children < -1) | (children >= N)
    if bad.any():
        raise ChildRangeError("child index outside [-1, N)")
    h = [-1] * N
    state = [0] * N          # 0 new, 1 on the recursion stack, 2 done

    def visit(v: int) -> int:
        if state[v] == 2:
            return h[v]
        if state[v] == 1:
            raise CycleError("cycle through node %d" % v)
        state[v] = 1
        best = -1
        for c in _kids(children, K, v):
            if c >= 0:
                best = max(best, visit(c))
        h[v] = best + 1
        state[v] = 2
        return h[v]

    with _deep_recursion(N + 1000):
        for v in range(N):
            visit(v)
    return np.array(h, dtype=np.int32)


def linearize(children: np.ndarray, K: int) -> Dict[str, np.ndarray]:
    """Definitional linearization.

    Rows are the nodes sorted by (height, id): level l occupies rows
    [level_offsets[l], level_offsets[l+1]).  ``child_rows[r*K+s]`` is the row
    of slot s of the node in row r, or -1.
    """
    children = np.asarray(children, dtype=np.int32)
    N = children.size // K
    h = heights(children, K)
    L = int(h.max()) + 1 if N > 0 else 0
    level_nodes = np.array(sorted(range(N), key=lambda v: (int(h[v]), v)), dtype=np.int32)
    counts = np.zeros(L, dtype=np.int64)
    for v in range(N):
        counts[h[v]] += 1
    level_offsets = np.zeros(L + 1, dtype=np.int32)
    for lvl in range(L):
        level_offsets[lvl + 1] = level_offsets[lvl] + counts[lvl]
    node_row = np.empty(N, dtype=np.int32)
    for r, v in enumerate(level_nodes):
        node_row[v] = r
    child_rows = np.full(N * K, -1, dtype=np.int32)
    for r, v in enumerate(level_nodes):
        for s, c in enumerate(_kids(children, K, int(v))):
            child_rows[r * K + s] = -1 if c < 0 else node_row[c]
    return {
        "height": h,
        "num_levels": np.int32(L),
        "level_offsets": level_offsets,
        "level_nodes": level_nodes,
        "node_row": node_row,
        "child_rows": child_rows,
    }


def dfs_batches(children: np.ndarray, K: int) -> List[List[int]]:
    """Batches of a tree forest in depth-first post-order (Sec. 4.2).

    The paper linearizes a tree by visiting it depth first and appending each
    node, once all of its children are done, to the batch of its height; leaves
    form batch 0.  Here the traversal is an explicit stack over the roots
    (nodes that fill no child slot) in ascending id: a frame is a node and the
    next child slot to descend into.  When a frame has no slot left, its
    node's height is one more than the largest child height (0 without
    children) and the node is appended to ``batches[height]``.

    Returns ``batches``: ``batches[h]`` lists the nodes of height h in the
    order the traversal completes them.
    """
    children = np.asarray(children, dtype=np.int32)
    N = children.size // K
    has_parent = np.zeros(N, dtype=bool)
    for c in children:
        if c >= 0:
            has_parent[c] = True
    height = np.full(N, -1, dtype=np.int64)
    batches: List[List[int]] = []
    for root in range(N):
        if has_parent[root]:
            continue
        stack = [[root, 0]]
        while stack:
            frame = stack[-1]
            node, slot = frame
            if slot < K:
                frame[1] = slot + 1
                c = int(children[node * K + slot])
                if c >= 0:
                    stack.append([c, 0])
                continue
            stack.pop()
            kid_heights = [int(height[c]) for c in _kids(children, K, node) if c >= 0]
            hgt = 1 + max(kid_heights) if kid_heights else 0
            height[node] = hgt
            while len(batches) <= hgt:
                batches.append([])
            batches[hgt].append(node)
    return batches


# ---------------------------------------------------------------------------
# Cells (per node, fp64)
# ---------------------------------------------------------------------------

def sigmoid(z: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-z))


class _Params:
    """fp32 inputs upcast once to fp64."""

    def __init__(self, cell: str, H: int, K: int, x_index=None, x_table=None, leaf_mat=None,
                 x=None, W=None, U=None, b=None, W_M=None):
        f = lambda a: None if a is None else np.asarray(a, dtype=np.float64)
        self.cell, self.H, self.K = cell, H, K
        self.x_index = None if x_index is None else np.asarray(x_index, dtype=np.int64)
        self.x_table, self.leaf_mat, self.x = f(x_table), f(leaf_mat), f(x)
        self.W, self.U, self.b, self.W_M = f(W), f(U), f(b), f(W_M)

    def input_row(self, v: int) -> np.ndarray:
        if self.x is not None:
            return self.x[v]
        i = -1 if self.x_index is None else int(self.x_index[v])
        return np.zeros(self.H) if i < 0 else self.x_table[i]


def _zero_state(p: _Params):
    H = p.H
    if p.cell in ("nary_treelstm", "childsum_treelstm"):
        return (np.zeros(H), np.zeros(H))
    if p.cell == "mvrnn":
        return (np.zeros(H), np.zeros((H, H)))
    return (np.zeros(H),)


def cell_apply(p: _Params, v: int, kids: Sequence[Optional[tuple]]):
    """State of node v from its child states (None = absent slot)."""
    H = p.H
    present = [k for k in kids if k is not None]
    is_leaf = len(present) == 0
    z = _zero_state(p)
    full = [k if k is not None else z for k in kids]

    if p.cell == "tree_rnn":
        if is_leaf:
            return (p.input_row(v).copy(),)
        hl, hr = full[0][0], full[1][0]
        return (np.tanh(p.W[:, :H] @ hl + p.W[:, H:] @ hr + p.b),)

    if p.cell == "nary_treelstm":
        if is_leaf:
            return (p.input_row(v).copy(), np.zeros(H))
        (hl, cl), (hr, cr) = full[0], full[1]
        Ul, Ur = p.U[0], p.U[1]
        a = [Ul[g] @ hl + Ur[g] @ hr + p.b[g] for g in range(5)]
        i, fl, fr, o = sigmoid(a[0]), sigmoid(a[1]), sigmoid(a[2]), sigmoid(a[3])
        u = np.tanh(a[4])
        c = i * u + fl * cl + fr * cr
        return (o * np.tanh(c), c)

    if p.cell == "childsum_treelstm":
        x = p.input_row(v)
        hsum = np.zeros(H)
        for hk, _ in present:
            hsum = hsum + hk
        Wi, Wf, Wo, Wu = p.W
        Ui, Uf, Uo, Uu = p.U
        bi, bf, bo, bu = p.b
        i = sigmoid(Wi @ x + Ui @ hsum + bi)
        o = sigmoid(Wo @ x + Uo @ hsum + bo)
        u = np.tanh(Wu @ x + Uu @ hsum + bu)
        c = i * u
        for hk, ck in present:
            fk = sigmoid(Wf @ x + Uf @ hk + bf)
            c = c + fk * ck
        return (o * np.tanh(c), c)

    if p.cell == "mvrnn":
        if is_leaf:
            i = -1 if p.x_index is None else int(p.x_index[v])
            if i < 0:
                return (np.zeros(H), np.zeros((H, H)))
            return (p.x_table[i].copy(), p.leaf_mat[i].copy())
        (a, A), (bb, B) = full[0], full[1]
        pvec = np.tanh(p.W @ np.concatenate([B @ a, A @ bb]))
        P = p.W_M @ np.concatenate([A, B], axis=0)
        return (pvec, P)

    if p.cell == "dagrnn":
        x = p.input_row(v)
        hu, hl = full[0][0], full[1][0]
        return (np.tanh(p.W @ x + p.U[0] @ hu + p.U[1] @ hl + p.b),)

    if p.cell in ("childsum_treegru", "simple_treegru"):
        x = p.input_row(v)
        Wz, Wr, Wh = p.W
        Uz, Ur, Uh = p.U
        bz, br, bh = p.b
        hsum = np.zeros(H)
        reset_sum = np.zeros(H)                  # sum over children of r_k * h_k
        for (hk,) in present:
            hsum = hsum + hk
            reset_sum = reset_sum + sigmoid(Wr @ x + Ur @ hk + br) * hk
        z = sigmoid(Wz @ x + Uz @ hsum + bz)
        cand = np.tanh(Wh @ x + Uh @ reset_sum + bh)
        if p.cell == "simple_treegru":
            return ((1.0 - z) * cand,)
        return (z * hsum + (1.0 - z) * cand,)

    raise ValueError("unknown cell %r" % p.cell)


def _as_arrays(cell: str, states: List[tuple]) -> Dict[str, np.ndarray]:
    out = {"h": np.stack([s[0] for s in states])}
    if cell in ("nary_treelstm", "childsum_treelstm"):
        out["c"] = np.stack([s[1] for s in states])
    if cell == "mvrnn":
        out["P"] = np.stack([s[1] for s in states])
    return out


def forward(cell: str, children: np.ndarray, K: int, H: int, **inputs) -> Dict[str, np.ndarray]:
    """Recursive memoized evaluation; states of every node, by node id."""
    children = np.asarray(children, dtype=np.int32)
    N = children.size // K
    heights(children, K)                          # validates range and acyclicity
    p = _Params(cell, H, K, **inputs)
    memo: Dict[int, tuple] = {}

    def state(v: int) -> tuple:
        if v in memo:
            return memo[v]
        kids = [None if c < 0 else state(c) for c in _kids(children, K, v)]
        memo[v] = cell_apply(p, v, kids)
        return memo[v]

    with _deep_recursion(N + 1000):
        states = [state(v) for v in range(N)]
    return _as_arrays(cell, states)


def forward_levels(cell: str, children: np.ndarray, K: int, H: int, order=None,
                   **inputs) -> Dict[str, np.ndarray]:
    """Iterative evaluation in a given child-before-parent node order.

    ``order`` defaults to the linearization's row order (level by level).
    Returns states by node id, like ``forward``.
    """
    children = np.asarray(children, dtype=np.int32)
    N = children.size // K
    if order is None:
        order = linearize(children, K)["level_nodes"]
    p = _Params(cell, H, K, **inputs)
    done: Dict[int, tuple] = {}
    for v in order:
        v = int(v)
        kids = []
        for c in _kids(children, K, v):
            if c < 0:
                kids.append(None)
            elif c not in done:
                raise ValueError("order evaluates node %d before its child %d" % (v, c))
            else:
                kids.append(done[c])
        done[v] = cell_apply(p, v, kids)
    return _as_arrays(cell, [done[v] for v in range(N)])


def forward_workload(wl) -> Dict[str, np.ndarray]:
    """Convenience wrapper over an ``inputs.Workload``-like object."""
    return forward(wl.cell, wl.children, wl.K, wl.H, x_index=wl.x_index, x_table=wl.x_table,
                   leaf_mat=wl.leaf_mat, x=wl.x, W=wl.W, U=wl.U, b=wl.b, W_M=wl.W_M)
