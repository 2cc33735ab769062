"""GPU forward parity: every cell against the fp64 oracle, element by element,
within 1e-4 max-abs and 1e-5 mean-abs, at the five full workloads (several
seeds) and at small ragged sizes; plus schedule variants, determinism and the
error paths."""
import numpy as np
import pytest
import torch

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import (announce, cached_oracle, cached_oracle_lin, cached_workload, compare_lin,
                               compare_states, need_gpu)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()
    yield
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_LIN_BLOCKS, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, 0)


def run(wl, groups=0):
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, groups)
    dw = DeviceWorkload(wl)
    dw.h.fill_(float("nan"))
    if dw.c is not None:
        dw.c.fill_(float("nan"))
    dw.step()
    st = dw.status_code()
    assert st == 0, "device status %d" % st
    return dw


@pytest.mark.parametrize("k", range(5))
@pytest.mark.parametrize("j", range(3))
def test_workload_parity(k, j, capsys):
    wl = cached_workload(k, j)
    announce("forward workload %d seed %d (%s N=%d)" % (k, j, wl.name, wl.N))
    dw = run(wl)
    compare_lin(dw.lin_host(), cached_oracle_lin(k, j), wl.K)
    got, ref = dw.states_by_node(), cached_oracle(k, j)
    if wl.cell == I.CELL_MVRNN:
        with capsys.disabled():          # shown in the test output even when the test passes
            report_mvrnn_depth(got, ref, cached_oracle_lin(k, j), "%s seed %d" % (wl.name, j))
    compare_states(got, ref, wl.name)


def report_mvrnn_depth(got, ref, lin, label):
    """Per-level max |P| and the level's max error relative to it, for P and
    p (ungraded).  The matrix state shrinks about 0.65x per level at
    W_M ~ U(+-0.1), so the absolute bound alone says little about the deep
    levels; this prints how the relative error behaves there."""
    height = lin["height"]
    print("[mvrnn-depth] %s: level, nodes, max|P|, max|dP|/max|P|, max|p|, max|dp|/max|p|" % label)
    for lvl in range(int(lin["num_levels"])):
        sel = height == lvl
        P_ref, P_got = ref["P"][sel], got["P"][sel]
        p_ref, p_got = ref["h"][sel], got["h"][sel]
        relP = float(np.abs(P_got - P_ref).max()) / max(float(np.abs(P_ref).max()), 1e-300)
        relp = float(np.abs(p_got - p_ref).max()) / max(float(np.abs(p_ref).max()), 1e-300)
        print("[mvrnn-depth] %2d %4d %.3e %.3e %.3e %.3e" % (lvl, int(sel.sum()), float(np.abs(P_ref).max()), relP,
                                                           float(np.abs(p_ref).max()), relp), flush=True)


SMALL = {
    "tree_rnn_h64": lambda s: I.tree_rnn_workload(s, n_leaves=int(np.random.default_rng(s).integers(1, 80)), H=64),
    "tree_rnn_h256": lambda s: I.tree_rnn_workload(s, n_leaves=37, H=256),
    "nary_h64": lambda s: I.nary_treelstm_workload(s, batch=4, H=64, vocab=50, leaf_lo=1, leaf_hi=30),
    "nary_h256": lambda s: I.nary_treelstm_workload(s, batch=3, H=256, vocab=50, leaf_lo=1, leaf_hi=25),
    "childsum_h64": lambda s: I.childsum_treelstm_workload(s, batch=4, H=64, vocab=50, node_lo=1, node_hi=60),
    "childsum_h256": lambda s: I.childsum_treelstm_workload(s, batch=3, H=256, vocab=50, node_lo=1, node_hi=40),
    "mvrnn": lambda s: I.mvrnn_workload(s, batch=4, d=64, leaf_lo=1, leaf_hi=30),
    "mvrnn_gain1": lambda s: I.mvrnn_workload(s, batch=3, d=64, leaf_lo=10, leaf_hi=40, wm_scale=0.153),
    "treegru_h64": lambda s: I.childsum_treegru_workload(s, batch=4, H=64, vocab=50, node_lo=1, node_hi=60),
    "treegru_h256": lambda s: I.childsum_treegru_workload(s, batch=3, H=256, vocab=50, node_lo=1, node_hi=40),
    "simple_treegru_h256": lambda s: I.childsum_treegru_workload(s, batch=3, H=256, vocab=50, node_lo=1,
                                                                 node_hi=40, simple=True),
    "dag_h64": lambda s: I.dagrnn_workload(s, n_grids=3, rows=7, cols=5, H=64),
    "dag_h256": lambda s: I.dagrnn_workload(s, n_grids=2, rows=9, cols=11, H=256),
    # the paper's large hidden sizes (h_l = 512; 128 for MV-RNN)
    "childsum_h512": lambda s: I.childsum_treelstm_workload(s, batch=3, H=512, vocab=50, node_lo=1, node_hi=40),
    "treegru_h512": lambda s: I.childsum_treegru_workload(s, batch=3, H=512, vocab=50, node_lo=1, node_hi=40),
    "simple_treegru_h512": lambda s: I.childsum_treegru_workload(s, batch=2, H=512, vocab=50, node_lo=1,
                                                                 node_hi=40, simple=True),
    "mvrnn_d128": lambda s: I.mvrnn_workload(s, batch=3, d=128, leaf_lo=1, leaf_hi=30),
    # W_M ~ U(+-sqrt(3)/16): unit gain at d = 128, so P stays O(0.1) through depth
    "mvrnn_d128_gain1": lambda s: I.mvrnn_workload(s, batch=2, d=128, leaf_lo=10, leaf_hi=40, wm_scale=0.108),
}


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("groups", [0, 1, 3])
def test_small_ragged(name, seed, groups):
    wl = SMALL[name](500 + seed)
    if wl.H == 512 and wl.cell != "tree_rnn" and groups > 2:
        groups = 2          # 128 hidden slices: two node groups fill the 256 compute units
    announce("small %s seed %d groups %d N=%d" % (name, seed, groups, wl.N))
    dw = run(wl, groups)
    compare_states(dw.states_by_node(), O.forward_workload(wl), name)


# Batches whose linearization does not fit the LDS structure cache: the
# kernels then stage each chunk of tiles' structure from global memory.
LARGE = {
    "tree_rnn_h256": lambda: I.tree_rnn_workload(31, n_leaves=1800, H=256),
    "nary_h256": lambda: I.nary_treelstm_workload(32, batch=120, H=256),
    "childsum_h256": lambda: I.childsum_treelstm_workload(33, batch=110, H=256),
    "childsum_h512": lambda: I.childsum_treelstm_workload(35, batch=60, H=512),
    "treegru_h512": lambda: I.childsum_treegru_workload(36, batch=60, H=512),
}


def test_mvrnn_d128_uncached_structure():
    """MV-RNN at d = 128 caches the structure in LDS only up to 640 rows
    ([A;B] takes 129 KB there): a batch of 40 trees runs uncached."""
    wl = I.mvrnn_workload(37, batch=40, d=128)
    assert wl.N > 640
    announce("uncached structure mvrnn d128 N=%d" % wl.N)
    dw = run(wl)
    compare_states(dw.states_by_node(), O.forward_workload(wl), wl.name)


@pytest.mark.parametrize("name", sorted(LARGE))
def test_uncached_structure(name):
    wl = LARGE[name]()
    assert wl.N > (2600 if wl.H < 512 else 1710), "must exceed the structure cache"
    announce("uncached structure %s N=%d" % (name, wl.N))
    dw = run(wl)
    compare_states(dw.states_by_node(), O.forward_workload(wl), name)


@pytest.mark.parametrize("groups", [0, 1])
def test_slice_units_change_only_the_schedule(groups):
    """Two hidden units per slice instead of four: the same contractions; at
    four units the u gate's rows are summed on the vector ALU (in another order
    than the MFMA tiles), so the states agree to fp32 rounding."""
    wl = cached_workload(1, groups)
    announce("slice units 2 vs default, seed %d, groups %d" % (groups, groups))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 0)
    ref = run(wl).states_by_node()
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 2)
    dw = run(wl, groups)
    assert C.cortex_last_grid(1) == 128 * (groups if groups else 2)
    got = dw.states_by_node()
    for key in ref:
        assert float(np.abs(ref[key] - got[key]).max()) <= 1e-5, key
    compare_states(got, cached_oracle(1, groups), wl.name)


def test_single_leaf_trees():
    for maker in (lambda: I.tree_rnn_workload(3, n_leaves=1, H=64),
                  lambda: I.nary_treelstm_workload(3, batch=1, H=256, leaf_lo=1, leaf_hi=1),
                  lambda: I.childsum_treelstm_workload(3, batch=1, H=256, node_lo=1, node_hi=1),
                  lambda: I.mvrnn_workload(3, batch=1, leaf_lo=1, leaf_hi=1),
                  lambda: I.dagrnn_workload(3, n_grids=1, rows=1, cols=1, H=256)):
        wl = maker()
        announce("single node %s" % wl.cell)
        dw = run(wl)
        compare_states(dw.states_by_node(), O.forward_workload(wl), wl.cell)


def test_caterpillar_deep_levels():
    """A 300-leaf caterpillar: 299 barrier-separated levels of one node."""
    children, is_leaf = I.forest_to_children([I.caterpillar(300, True)], 2)
    wl = I.nary_treelstm_workload(9, batch=1, H=256)
    rng = np.random.default_rng(9)
    wl.children = children
    wl.x_index = np.where(is_leaf, rng.integers(0, 1000, is_leaf.size), -1).astype(np.int32)
    announce("caterpillar 300")
    dw = run(wl)
    compare_states(dw.states_by_node(), O.forward_workload(wl), "caterpillar")


def test_dag_input_with_shared_children():
    """Tree cells accept DAGs: a node may be the child of several nodes."""
    rng = np.random.default_rng(3)
    ch = I.random_dag(rng, 400, 2, p_absent=0.2)
    wl = I.tree_rnn_workload(4, n_leaves=2, H=64)
    wl.children = ch
    ch2 = ch.reshape(-1, 2)
    leaf = (ch2 < 0).all(1)
    wl.x_table = rng.standard_normal((int(leaf.sum()), 64)).astype(np.float32)
    wl.x_index = np.where(leaf, np.cumsum(leaf) - 1, -1).astype(np.int32)
    announce("tree_rnn over random DAG")
    dw = run(wl)
    compare_states(dw.states_by_node(), O.forward_workload(wl), "dag-tree_rnn")


@pytest.mark.parametrize("k", range(5))
def test_deterministic(k):
    wl = cached_workload(k, 0)
    announce("determinism workload %d" % k)
    dw = run(wl)
    first = dw.states_by_node()
    for _ in range(5):
        dw.step()
        assert dw.status_code() == 0
        again = dw.states_by_node()
        for key in first:
            np.testing.assert_array_equal(again[key], first[key])


def test_failed_linearization_makes_forward_a_noop():
    wl = I.nary_treelstm_workload(5, batch=2, H=256)
    wl.children = wl.children.copy()
    wl.children[-1] = wl.N - 1            # root becomes its own child: a cycle
    announce("cycle -> forward no-op")
    dw = DeviceWorkload(wl)
    dw.h.fill_(float("nan"))
    dw.step()
    assert dw.status_code() == C.CORTEX_ST_CYCLE
    assert torch.isnan(dw.h).all()


def test_input_index_out_of_range():
    wl = I.nary_treelstm_workload(6, batch=2, H=256)
    leaf = np.where(wl.x_index >= 0)[0][0]
    wl.x_index = wl.x_index.copy()
    wl.x_index[leaf] = 5000                # beyond the 1000-row table
    announce("x_index out of range")
    dw = DeviceWorkload(wl)
    dw.step()
    assert dw.status_code() == C.CORTEX_ST_INPUT_RANGE


def test_host_errors_enqueue_nothing():
    wl = cached_workload(1, 0)
    dw = DeviceWorkload(wl)
    # unsupported hidden size
    rc = C.cortex_tree_forward(C.CORTEX_NARY_TREELSTM, 100, dw.lin, dw.x_table, dw.x_rows, dw.x_index, None,
                               U=dw.U, b=dw.b, h=dw.h, c_or_P=dw.c, status=dw.status, ws=dw.ws_fwd)
    assert rc == C.CORTEX_E_INVAL
    # workspace too small
    small = torch.zeros(16, dtype=torch.uint8, device="cuda")
    rc = C.cortex_tree_forward(C.CORTEX_NARY_TREELSTM, 256, dw.lin, dw.x_table, dw.x_rows, dw.x_index, None,
                               U=dw.U, b=dw.b, h=dw.h, c_or_P=dw.c, status=dw.status, ws=small)
    assert rc == C.CORTEX_E_WORKSPACE
    # more node groups than can be co-resident
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, 100000)
    rc = C.cortex_tree_forward(C.CORTEX_NARY_TREELSTM, 256, dw.lin, dw.x_table, dw.x_rows, dw.x_index, None,
                               U=dw.U, b=dw.b, h=dw.h, c_or_P=dw.c, status=dw.status, ws=dw.ws_fwd)
    assert rc == C.CORTEX_E_TOO_LARGE


@pytest.mark.parametrize("units,groups", [(64, 0), (64, 8), (64, 5), (16, 0), (16, 2), (0, 0)])
def test_dag_slice_widths(units, groups):
    """DAG-RNN at H = 256 under both slice widths (64 and 16 units; 0 = the
    size-based default, 16 units at this size) and grids that do (multiples
    of 32 workgroups) and do not use the XCD-grouped block order; each
    against the oracle."""
    wl = I.dagrnn_workload(77, n_grids=5, rows=13, cols=9, H=256)
    announce("dag slice units %d groups %d N=%d" % (units, groups, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, units)
    dw = run(wl, groups)
    S = 4 if units == 64 else 16
    assert C.cortex_last_grid(1) == S * (groups if groups else 256 // S)
    compare_states(dw.states_by_node(), O.forward_workload(wl), "dag units %d" % units)


@pytest.mark.parametrize("groups", [2, 3])
def test_dag_two_tile_steps_ragged(groups):
    """64-unit DAG-RNN slices with few node groups, so most steps carry two
    tiles (tile 1's child fragments are requested during tile 0's recurrent
    part and waited for on their own) and levels end in ragged tiles; ten
    20x15 grids, against the oracle."""
    wl = I.dagrnn_workload(79 + groups, n_grids=10, rows=20, cols=15, H=256)
    announce("dag two-tile steps groups %d N=%d" % (groups, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 64)
    dw = run(wl, groups)
    assert C.cortex_last_grid(1) == 4 * groups
    compare_states(dw.states_by_node(), O.forward_workload(wl), "dag two-tile groups %d" % groups)


@pytest.mark.parametrize("groups,n_grids,side", [(16, 8, 24), (64, 3, 20), (2, 6, 32), (5, 4, 12)])
def test_dag_half_steps(groups, n_grids, side):
    """Levels of at most groups/2 tiles run as half steps (two groups per
    tile, 32 units each): 8 grids of 24x24 over 16 groups mix half levels
    (up to 128 rows) with whole ones, so groups change kind of step at
    either parity of their step lists; 3 grids of 20x20 over 64 groups are
    half steps throughout; 2 groups over 6 grids of 32x32 overflow the step
    list, so the half steps of the one-tile levels fall in its first and
    last chunks;
    an odd group count (5) never splits.  Ragged tiles throughout; against
    the oracle."""
    wl = I.dagrnn_workload(90 + groups, n_grids=n_grids, rows=side, cols=side, H=256)
    announce("dag half steps groups %d N=%d" % (groups, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 64)
    dw = run(wl, groups)
    assert C.cortex_last_grid(1) == 4 * groups
    compare_states(dw.states_by_node(), O.forward_workload(wl), "dag half steps groups %d" % groups)


def test_dag_tile_list_overflow():
    """One node group over 6 grids of 32x32: the group's steps (several per
    level) exceed the per-workgroup step list many times over, so the kernel
    lists and runs them a chunk at a time; against the oracle."""
    wl = I.dagrnn_workload(78, n_grids=6, rows=32, cols=32, H=256)
    announce("dag tile-list overflow N=%d" % wl.N)
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 64)
    dw = run(wl, 1)
    assert C.cortex_last_grid(1) == 4
    compare_states(dw.states_by_node(), O.forward_workload(wl), "dag overflow")


@pytest.mark.parametrize("unroll", [0, 1])
@pytest.mark.parametrize("n_leaves", [1, 2, 7, 160, 161, 230])
def test_tree_rnn_h64_lds_limit(n_leaves, unroll):
    """TreeRNN at H = 64 runs in one workgroup with every state in LDS up to
    320 rows (160 leaves: 319 rows) and one workgroup per tree beyond (here
    one tree: one busy workgroup); the unroll knob at 1 forces the
    level-parallel slices.  Both sides of the limit against the oracle."""
    wl = I.tree_rnn_workload(600 + n_leaves, n_leaves=n_leaves, H=64)
    announce("tree_rnn h64 %d leaves N=%d unroll %d" % (n_leaves, wl.N, unroll))
    C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, unroll)
    try:
        dw = run(wl)
        if unroll == 0:
            assert C.cortex_last_grid(1) == (1 if wl.N <= 320 else min(256, (wl.N + 15) // 16))
        compare_states(dw.states_by_node(), O.forward_workload(wl), "tree_rnn %d leaves" % n_leaves)
    finally:
        C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 0)


_ORACLE_MEMO = {}


def _oracle_of(name, wl):
    """fp64 oracle states of a schedule test's workload (computed once per
    case name and workload: the parametrized modes share it)."""
    key = (name, wl.name, wl.N)
    if key not in _ORACLE_MEMO:
        _ORACLE_MEMO[key] = O.forward_workload(wl)
    return _ORACLE_MEMO[key]


LEVEL_SYNC_CASES = {
    "treegru": (lambda: I.childsum_treegru_workload(44, batch=4, H=256), 0),
    "nary": (lambda: cached_workload(1, 0), 0),
    "childsum": (lambda: cached_workload(2, 0), 0),
    "tree_rnn_h256": (lambda: I.tree_rnn_workload(41, n_leaves=37, H=256), 0),
    "dag_h256_units16": (lambda: I.dagrnn_workload(42, n_grids=3, rows=9, cols=7, H=256), 16),
    "dag_h256_units64": (lambda: I.dagrnn_workload(43, n_grids=3, rows=9, cols=7, H=256), 64),
}


@pytest.mark.parametrize("name", sorted(LEVEL_SYNC_CASES))
@pytest.mark.parametrize("mode", [1, 2])
def test_level_sync_modes_change_only_the_schedule(name, mode):
    """The ablation modes (a device-wide barrier after every level; one
    launch per level) run the same arithmetic in the same order as the
    default per-datum waits, so the states are bitwise identical; a kernel
    without the mode rejects it on the host."""
    make, units = LEVEL_SYNC_CASES[name]
    wl = make()
    announce("level sync mode %d %s N=%d" % (mode, name, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, units)
    ref = run(wl).states_by_node()
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, mode)
    if name == "dag_h256_units64" and mode == 1:
        dw = DeviceWorkload(wl)
        dw.linearize()
        with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
            dw.forward()
        return
    got = run(wl).states_by_node()
    oracle = _oracle_of(name, wl)
    compare_states(ref, oracle, "%s default" % name)
    compare_states(got, oracle, "%s level sync %d" % (name, mode))
    for key in ref:
        assert np.array_equal(ref[key], got[key]), key


ABLATE_CASES = {
    "nary": (lambda: cached_workload(1, 0), 0, 3),
    "nary_units2": (lambda: I.nary_treelstm_workload(48, batch=4, H=256), 2, 3),
    "nary_uncached": (lambda: I.nary_treelstm_workload(32, batch=120, H=256), 0, 3),
    "tree_rnn_h256": (lambda: I.tree_rnn_workload(41, n_leaves=37, H=256), 0, 3),
    "tree_rnn_h512": (lambda: I.tree_rnn_workload(49, n_leaves=23, H=512), 0, 3),
    "dag_h256_units16": (lambda: I.dagrnn_workload(42, n_grids=3, rows=9, cols=7, H=256), 16, 1),
    "dag_h256_units64": (lambda: I.dagrnn_workload(43, n_grids=3, rows=9, cols=7, H=256), 64, 4),
}


@pytest.mark.parametrize("name", sorted(ABLATE_CASES))
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_ablations_change_only_the_schedule(name, bits):
    """Weights read from memory at every tile (bit 0) and leaf states staged
    and waited for (bit 1) feed the same values to the same contraction
    order, so the states are bitwise identical; the hoisted input products
    (bit 2, DAG-RNN with 64-unit slices) add the same terms in another order,
    so they meet the oracle only.  A kernel without the ablation rejects it
    on the host."""
    make, units, supported = ABLATE_CASES[name]
    wl = make()
    announce("ablate %d %s N=%d" % (bits, name, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, units)
    ref = run(wl).states_by_node()
    C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, bits)
    if bits & ~supported:
        dw = DeviceWorkload(wl)
        dw.linearize()
        with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
            dw.forward()
        assert dw.status_code() == 0
        return
    oracle = _oracle_of(name, wl)
    compare_states(ref, oracle, "%s default" % name)
    for sync in (0, 2):
        C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, sync)
        got = run(wl).states_by_node()
        compare_states(got, oracle, "%s ablate %d level sync %d" % (name, bits, sync))
        if bits & 4:
            continue
        for key in ref:
            assert np.array_equal(ref[key], got[key]), (key, sync)


def test_hoisted_input_products_full_grid():
    """The 64-grid DAG-RNN batch with its input products hoisted into one
    matrix product before the level loop (CORTEX_KNOB_ABLATE bit 2) against
    the oracle, element by element."""
    wl = I.make_workload(4)
    announce("hoisted input products, %s N=%d" % (wl.name, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, 4)
    got = run(wl).states_by_node()
    compare_states(got, _oracle_of("w4", wl), "%s hoisted" % wl.name)


@pytest.mark.parametrize("k", [0, 2, 3])
def test_ablations_unsupported(k):
    """Kernels other than the slice kernel have no ablation switches."""
    wl = cached_workload(k, 0)
    announce("ablate unsupported on workload %d" % k)
    C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, 1)
    dw = DeviceWorkload(wl)
    dw.linearize()
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0


@pytest.mark.parametrize("k", [0, 3])
@pytest.mark.parametrize("mode", [1, 2])
def test_level_sync_modes_unsupported(k, mode):
    """TreeRNN H = 64 (states in LDS) and MV-RNN have no ablation modes."""
    wl = cached_workload(k, 0)
    announce("level sync mode %d unsupported on workload %d" % (mode, k))
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, mode)
    dw = DeviceWorkload(wl)
    dw.linearize()
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0


TREEGRU_SPLIT_CASES = {
    "treegru_h256_b4": lambda: I.childsum_treegru_workload(44, batch=4, H=256),
    "simple_treegru_h256_b10": lambda: I.childsum_treegru_workload(45, batch=10, H=256, simple=True),
    "treegru_h64_b10": lambda: I.childsum_treegru_workload(46, batch=10, H=64),
    "treegru_h256_uncached": lambda: I.childsum_treegru_workload(47, batch=110, H=256),
}


@pytest.mark.parametrize("name", sorted(TREEGRU_SPLIT_CASES))
def test_treegru_phase_barrier_mode(name):
    """LEVEL_SYNC 3 (a device-wide barrier between the reset sums and the
    candidate, and another closing the level) keeps phase-A values in the
    workspace across the barrier; the states are bitwise those of the
    default schedule."""
    wl = TREEGRU_SPLIT_CASES[name]()
    announce("treegru phase barrier %s N=%d" % (name, wl.N))
    ref = run(wl).states_by_node()
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 3)
    got = run(wl).states_by_node()
    oracle = _oracle_of(name, wl)
    compare_states(ref, oracle, "%s default" % name)
    compare_states(got, oracle, "%s phase barrier" % name)
    for key in ref:
        assert np.array_equal(ref[key], got[key]), key


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
def test_phase_barrier_mode_needs_two_exchanges(k):
    """Only the TreeGRU kernels have a second exchange per level; the other
    forwards reject LEVEL_SYNC 3 on the host and enqueue nothing."""
    wl = cached_workload(k, 0)
    announce("level sync mode 3 unsupported on workload %d" % k)
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 3)
    dw = DeviceWorkload(wl)
    dw.linearize()
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0


@pytest.mark.parametrize("simple", [False, True])
@pytest.mark.parametrize("seed", [0, 1])
def test_treegru_batch10_parity(simple, seed):
    """Child-sum TreeGRU and SimpleTreeGRU, H = 256, a batch of 10 SST-sized
    random trees (arity 1-4), against the oracle."""
    wl = I.childsum_treegru_workload(I.BASE_SEED + 50 + seed, batch=10, H=256, simple=simple)
    announce("%s seed %d N=%d" % (wl.name, seed, wl.N))
    dw = run(wl)
    compare_lin(dw.lin_host(), O.linearize(wl.children, wl.K), wl.K)
    compare_states(dw.states_by_node(), O.forward_workload(wl), wl.name)


def test_treegru_uncached_structure():
    """A TreeGRU batch too large for the LDS structure cache."""
    wl = I.childsum_treegru_workload(34, batch=110, H=256)
    assert wl.N > 2600
    announce("treegru uncached N=%d" % wl.N)
    dw = run(wl)
    compare_states(dw.states_by_node(), O.forward_workload(wl), wl.name)
