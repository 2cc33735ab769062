"""cortex_tree_infer and cortex_dag_infer: linearization and forward in one call.  For the cells
with a fused instance (TreeRNN, N-ary and child-sum TreeLSTM, TreeGRU cells,
MV-RNN at d = 64, DAG-RNN with 16-unit slices)
it is one launch in which every workgroup linearizes the batch itself;
its linearization must be bit-exact and its states bitwise those of
cortex_linearize followed by cortex_tree_forward (the same contraction in the
same order), and both match the oracle.  Other cells, larger batches and
non-default schedule knobs take the two launches."""
import dataclasses

import numpy as np
import pytest

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import (announce, cached_oracle, cached_workload, compare_lin, compare_states,
                               need_gpu)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()
    yield
    for k in (C.CORTEX_KNOB_FWD_NODE_GROUPS, C.CORTEX_KNOB_FWD_SLICE_UNITS, C.CORTEX_KNOB_LEVEL_SYNC,
              C.CORTEX_KNOB_ABLATE, C.CORTEX_KNOB_LIN_BLOCKS, C.CORTEX_KNOB_TREE_UNROLL):
        C.cortex_set_knob(k, 0)


def _states(dw):
    dw.h.fill_(float("nan"))
    if dw.c is not None:
        dw.c.fill_(float("nan"))


def infer_and_two_calls(wl, groups=0):
    """(infer's lin, states, linearizer grid) and (two calls' lin, states)."""
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, groups)
    a = DeviceWorkload(wl)
    _states(a)
    a.lin.level_nodes.fill_(-7)
    a.infer()
    assert a.status_code() == 0
    grid0 = C.cortex_last_grid(0)
    b = DeviceWorkload(wl)
    _states(b)
    b.step_two_calls()
    assert b.status_code() == 0
    return (a.lin_host(), a.states_by_node(), grid0), (b.lin_host(), b.states_by_node())


FUSED = {
    "nary_h256_b10": lambda: cached_workload(1, 0),
    "nary_h256_b10_seed1": lambda: cached_workload(1, 1),
    "nary_h64_ragged": lambda: I.nary_treelstm_workload(61, batch=7, H=64, vocab=50, leaf_lo=1, leaf_hi=30),
    "nary_h256_single_leaf": lambda: I.nary_treelstm_workload(62, batch=1, H=256, leaf_lo=1, leaf_hi=1),
    "nary_h256_b25": lambda: I.nary_treelstm_workload(63, batch=25, H=256),
    "treefc_h256_b1": lambda: I.treefc_workload(64, batch=1, H=256),
    "treefc_h512_b4": lambda: I.treefc_workload(65, batch=4, H=512),
    "tree_rnn_h256_relabeled": lambda: _relabeled(I.tree_rnn_workload(66, n_leaves=57, H=256), 66),
    "tree_rnn_h64_1x32": lambda: cached_workload(0, 0),
    "tree_rnn_h64_ragged": lambda: I.tree_rnn_workload(67, n_leaves=150, H=64),
    "childsum_h256_b10": lambda: cached_workload(2, 0),
    "childsum_h64_ragged": lambda: I.childsum_treelstm_workload(68, batch=5, H=64, vocab=50, node_lo=1, node_hi=60),
    "childsum_h512_b3": lambda: I.childsum_treelstm_workload(69, batch=3, H=512),
    "treegru_h256_b10": lambda: I.childsum_treegru_workload(70, batch=10, H=256),
    "simple_treegru_h64": lambda: I.childsum_treegru_workload(80, batch=4, H=64, simple=True),
    "treegru_h512_b2": lambda: I.childsum_treegru_workload(81, batch=2, H=512),
    "mvrnn_d64_b10": lambda: cached_workload(3, 0),
    "mvrnn_d64_ragged": lambda: I.mvrnn_workload(82, batch=4, d=64, leaf_lo=1, leaf_hi=30),
    "dag_h256_10x10": lambda: I.paper_grid_workload("dagrnn", 1, "s"),
    "dag_h256_10x10_b10": lambda: I.paper_grid_workload("dagrnn", 10, "s"),
    "dag_h64_ragged": lambda: I.dagrnn_workload(83, n_grids=3, rows=7, cols=5, H=64),
    "dag_h512_ragged": lambda: I.dagrnn_workload(84, n_grids=2, rows=9, cols=11, H=512),
}

ORACLE_CACHED = {"nary_h256_b10": (1, 0), "nary_h256_b10_seed1": (1, 1), "tree_rnn_h64_1x32": (0, 0),
                 "childsum_h256_b10": (2, 0), "mvrnn_d64_b10": (3, 0)}


def _relabeled(wl, seed):
    """The same batch with node ids shuffled (inputs follow their nodes)."""
    perm = np.random.default_rng(seed).permutation(wl.N).astype(np.int32)
    x_index = np.empty_like(wl.x_index)
    x_index[perm] = wl.x_index
    return dataclasses.replace(wl, name=wl.name + "_relabeled", children=I.relabel(wl.children, wl.K, perm),
                               x_index=x_index)


@pytest.mark.parametrize("name", sorted(FUSED))
def test_fused_launch_matches_two_calls_and_oracle(name):
    wl = FUSED[name]()
    announce("infer fused %s N=%d" % (name, wl.N))
    (lin_a, st_a, grid0), (lin_b, st_b) = infer_and_two_calls(wl)
    assert grid0 == 0, "the fused launch was not taken"
    ref_lin = O.linearize(wl.children, wl.K)
    compare_lin(lin_a, ref_lin, wl.K)
    compare_lin(lin_b, ref_lin, wl.K)
    for key in st_b:
        assert np.array_equal(st_a[key], st_b[key]), key
    ref = cached_oracle(*ORACLE_CACHED[name]) if name in ORACLE_CACHED else O.forward_workload(wl)
    compare_states(st_a, ref, name)


def test_dag_64_grids_two_launches():
    """The 65,536-node grid batch: cortex_dag_infer takes the two launches."""
    wl = cached_workload(4, 0)
    announce("dag infer 64 grids N=%d" % wl.N)
    dw = DeviceWorkload(wl)
    _states(dw)
    dw.infer()
    assert dw.status_code() == 0
    assert C.cortex_last_grid(0) >= 1
    compare_states(dw.states_by_node(), cached_oracle(4, 0), wl.name)


@pytest.mark.parametrize("grids", [128, 300])
def test_dag_large_batches(grids):
    """Batches beyond the headline's 64 grids of 32x32 through
    cortex_dag_infer: at 128 grids (131,072 nodes) each node group has about
    95 steps, more than its step list holds, so it runs them in listed
    chunks; at 300 grids (307,200 nodes) the linearizer also takes its
    instance with two workgroups per compute unit.  Every state against the
    oracle."""
    wl = I.dagrnn_workload(I.BASE_SEED + 3000 + grids, n_grids=grids)
    announce("dag infer %d grids N=%d" % (grids, wl.N))
    dw = DeviceWorkload(wl)
    _states(dw)
    dw.infer()
    assert dw.status_code() == 0
    compare_states(dw.states_by_node(), O.forward_workload(wl), wl.name)


@pytest.mark.parametrize("groups", [1, 3])
def test_fused_launch_node_groups(groups):
    wl = cached_workload(1, 2)
    announce("infer fused groups %d" % groups)
    (lin_a, st_a, grid0), (_, st_b) = infer_and_two_calls(wl, groups)
    assert grid0 == 0
    assert C.cortex_last_grid(1) == 64 * groups
    for key in st_b:
        assert np.array_equal(st_a[key], st_b[key]), key


TWO_LAUNCH = {
    "tree_rnn_h64_over_320": (lambda: I.tree_rnn_workload(71, n_leaves=200, H=64), None),
    "tree_rnn_h64_unroll": (lambda: I.tree_rnn_workload(72, n_leaves=40, H=64), (C.CORTEX_KNOB_TREE_UNROLL, 2)),
    # d = 128: [A; B] alone takes 129 KB of LDS, the linearization does not fit beside it
    "mvrnn_d128": (lambda: I.mvrnn_workload(73, batch=3, d=128), None),
    "treegru_h256_phase_barrier": (lambda: I.childsum_treegru_workload(74, batch=3, H=256),
                                   (C.CORTEX_KNOB_LEVEL_SYNC, 3)),
    "nary_h256_over_2048": (lambda: I.nary_treelstm_workload(75, batch=90, H=256), None),
    # fused LDS at H = 256: 84 KB of weights and partial sums + 48 N + 10.5 KB
    "nary_h256_beyond_lds": (lambda: I.nary_treelstm_workload(63, batch=40, H=256), None),
    "nary_h256_units2": (lambda: I.nary_treelstm_workload(76, batch=5, H=256), (C.CORTEX_KNOB_FWD_SLICE_UNITS, 2)),
    "nary_h256_level_sync": (lambda: I.nary_treelstm_workload(77, batch=5, H=256), (C.CORTEX_KNOB_LEVEL_SYNC, 1)),
    "dag_h256_units64": (lambda: I.dagrnn_workload(85, n_grids=3, rows=9, cols=7, H=256),
                         (C.CORTEX_KNOB_FWD_SLICE_UNITS, 64)),
}


@pytest.mark.parametrize("name", sorted(TWO_LAUNCH))
def test_two_launch_fallback(name):
    make, knob = TWO_LAUNCH[name]
    wl = make()
    announce("infer two launches %s N=%d" % (name, wl.N))
    if knob:
        C.cortex_set_knob(*knob)
    dw = DeviceWorkload(wl)
    _states(dw)
    dw.infer()
    assert dw.status_code() == 0
    assert C.cortex_last_grid(0) >= 1, "expected the separate linearizer launch"
    compare_lin(dw.lin_host(), O.linearize(wl.children, wl.K), wl.K)
    compare_states(dw.states_by_node(), O.forward_workload(wl), name)


def _with_children(wl, children):
    return dataclasses.replace(wl, children=np.asarray(children, dtype=np.int32))


@pytest.mark.parametrize("cell", ["nary", "childsum"])
@pytest.mark.parametrize("case", ["range_high", "range_low", "cycle"])
def test_fused_launch_errors(cell, case):
    """Invalid structures set the status and write no states."""
    if cell == "nary":
        base = I.nary_treelstm_workload(78, batch=1, H=256, leaf_lo=4, leaf_hi=4)     # 7 nodes, K = 2
    else:
        base = I.childsum_treelstm_workload(79, batch=1, H=256, node_lo=9, node_hi=9)  # K = 4
    ch = base.children.copy()
    if case == "range_high":
        ch[np.nonzero(ch >= 0)[0][0]] = 99
        want = C.CORTEX_ST_CHILD_RANGE
    elif case == "range_low":
        ch[np.nonzero(ch >= 0)[0][0]] = -3
        want = C.CORTEX_ST_CHILD_RANGE
    else:
        K = base.K
        root = int(np.nonzero((ch.reshape(-1, K) >= 0).any(1))[0][-1])
        leaf = int(np.nonzero((ch.reshape(-1, K) < 0).all(1))[0][0])
        ch[leaf * K] = root                       # a leaf now points at the root: a cycle
        want = C.CORTEX_ST_CYCLE
    wl = _with_children(base, ch)
    announce("infer fused error %s %s" % (cell, case))
    dw = DeviceWorkload(wl)
    dw.h.fill_(7.0)
    dw.infer()
    assert dw.status_code() == want
    assert C.cortex_last_grid(0) == 0
    assert bool((dw.h == 7.0).all())
    dw.reset_status()
    ok = DeviceWorkload(base)
    ok.infer()
    assert ok.status_code() == 0
