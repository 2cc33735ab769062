"""Unrolled TreeRNN at H = 64 (Secs. 3.1, 7.4): one workgroup evaluates each
tree from its leaves to its root.  Parity against the oracle on batches of
trees, the edge cases of the tree-to-workgroup assignment (single-node trees,
trees interleaved in id order, workgroups owning several trees, more rows
than LDS holds, nodes with several parents), bitwise agreement with the
single-workgroup kernel, and the host-side limits."""
import numpy as np
import pytest

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import announce, compare_lin, compare_states, need_gpu

pytestmark = pytest.mark.gpu

FOREST_MAX_ROWS = 2048


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()
    yield
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 0)


def run(wl, unroll, groups=0):
    C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, unroll)
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, groups)
    dw = DeviceWorkload(wl)
    dw.h.fill_(float("nan"))
    dw.step()
    st = dw.status_code()
    assert st == 0, "device status %d" % st
    return dw


def shared_children_workload(seed, N):
    """TreeRNN over a random DAG (nodes with several parents), H = 64."""
    rng = np.random.default_rng(seed)
    ch = I.random_dag(rng, N, 2)
    is_leaf = (ch.reshape(N, 2) < 0).all(axis=1)
    x_index = np.full(N, -1, dtype=np.int32)
    x_index[is_leaf] = np.arange(int(is_leaf.sum()), dtype=np.int32)
    leaves = rng.standard_normal((int(is_leaf.sum()), 64)).astype(np.float32)
    W = rng.uniform(-0.1, 0.1, (64, 128)).astype(np.float32)
    return I.Workload("tree_rnn_h64_dag%d" % N, I.CELL_TREE_RNN, 64, 2, ch, x_index=x_index, x_table=leaves, W=W,
                      b=np.zeros(64, dtype=np.float32))


FOREST = {
    "b10x32": lambda: I.tree_rnn_forest_workload(70, batch=10),
    "b30_1to60_shuffled": lambda: I.tree_rnn_forest_workload(71, batch=30, leaf_lo=1, leaf_hi=60, shuffle=True),
    "b64_1to3_shuffled": lambda: I.tree_rnn_forest_workload(72, batch=64, leaf_lo=1, leaf_hi=3, shuffle=True),
    "b4_200to250": lambda: I.tree_rnn_forest_workload(73, batch=4, leaf_lo=200, leaf_hi=250),
    "b1x1000": lambda: I.tree_rnn_forest_workload(74, batch=1, leaf_lo=1000, leaf_hi=1000),
    "dag200": lambda: shared_children_workload(75, 200),
    "dag900": lambda: shared_children_workload(76, 900),
}


@pytest.mark.parametrize("name", sorted(FOREST))
@pytest.mark.parametrize("unroll,groups", [(2, 0), (2, 1), (2, 3), (1, 0)])
def test_tree_rnn_unroll_parity(name, unroll, groups):
    """One workgroup per tree (grid from the batch size, one workgroup for
    everything, three workgroups sharing the trees) and the level-parallel
    slices, each against the oracle."""
    wl = FOREST[name]()
    assert wl.N <= FOREST_MAX_ROWS
    announce("tree_rnn unroll %d groups %d %s N=%d" % (unroll, groups, name, wl.N))
    dw = run(wl, unroll, groups)
    if unroll == 2:
        assert C.cortex_last_grid(1) == (groups if groups else min(256, (wl.N + 15) // 16))
    compare_lin(dw.lin_host(), O.linearize(wl.children, wl.K), wl.K)
    compare_states(dw.states_by_node(), O.forward_workload(wl), "%s unroll %d groups %d" % (name, unroll, groups))


@pytest.mark.parametrize("name", ["b64_1to3_shuffled", "dag200", "b30_1to60_shuffled", "b4_200to250"])
def test_unrolled_states_are_bitwise_those_of_one_workgroup(name):
    """Per node the unrolled kernel runs the arithmetic of the single-
    workgroup kernel in the same order, whether its states sit in LDS or in
    the output rows, so every assignment gives bitwise identical states."""
    wl = FOREST[name]()
    announce("tree_rnn unroll bitwise %s N=%d" % (name, wl.N))
    ref = run(wl, 2, 1).states_by_node()["h"]
    for unroll, groups in ((2, 0), (2, 2), (2, 7), (0, 0)):
        got = run(wl, unroll, groups).states_by_node()["h"]
        assert np.array_equal(ref, got), (unroll, groups)


def test_unroll_limit():
    """Above 2048 nodes the unrolled kernel is refused on the host (nothing
    enqueued); the default then takes the level-parallel slices."""
    wl = I.tree_rnn_forest_workload(77, batch=32, leaf_lo=1, leaf_hi=64)
    assert wl.N > FOREST_MAX_ROWS
    announce("tree_rnn unroll limit N=%d" % wl.N)
    C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 2)
    dw = DeviceWorkload(wl)
    dw.linearize()
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0
    dw = run(wl, 0)
    compare_states(dw.states_by_node(), O.forward_workload(wl), "tree_rnn above the unroll limit")


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_unrolled_kernel_has_no_level_sync_modes(mode):
    wl = FOREST["b10x32"]()
    announce("tree_rnn unroll with level sync %d" % mode)
    C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 2)
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, mode)
    try:
        dw = DeviceWorkload(wl)
        dw.linearize()
        with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
            dw.forward()
        assert dw.status_code() == 0
    finally:
        C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 0)
