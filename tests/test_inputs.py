"""Seeded generators: determinism and the structure statistics of the workloads."""
import numpy as np
import pytest

from paper_2011_01383_amd import inputs as I


@pytest.mark.parametrize("k", range(5))
def test_deterministic(k):
    a, b = I.make_workload(k), I.make_workload(k)
    for f in ("children", "x_index", "x_table", "leaf_mat", "x", "W", "U", "b", "W_M"):
        va, vb = getattr(a, f), getattr(b, f)
        assert (va is None) == (vb is None)
        if va is not None:
            assert va.dtype in (np.int32, np.float32)
            np.testing.assert_array_equal(va, vb)
    c = I.make_workload(k, 1)
    if k != 4:      # the grid structure is fixed; only its data depend on the seed
        assert c.children.size != a.children.size or (c.children != a.children).any()


def test_tree_rnn_shape():
    wl = I.make_workload(0)
    assert (wl.N, wl.K, wl.H) == (63, 2, 64)
    assert wl.x_table.shape == (32, 64) and wl.W.shape == (64, 128)
    assert (wl.b == 0).all() and np.abs(wl.W).max() <= 0.1
    ch = wl.children.reshape(-1, 2)
    assert ((ch[:, 0] >= 0) == (ch[:, 1] >= 0)).all()          # full binary
    assert int((ch[:, 0] < 0).sum()) == 32


@pytest.mark.parametrize("k", [1, 3])
def test_binary_forests(k):
    wl = I.make_workload(k)
    ch = wl.children.reshape(-1, 2)
    n_leaf = int((ch[:, 0] < 0).sum())
    n_int = int((ch[:, 0] >= 0).sum())
    assert n_leaf == n_int + 10                                # 10 full binary trees
    assert 10 * 10 <= n_leaf <= 10 * 40
    # post-order numbering: children precede parents
    for v in range(ch.shape[0]):
        assert all(c < v for c in ch[v] if c >= 0)


def test_childsum_forest():
    wl = I.make_workload(2)
    assert wl.K == 4 and wl.x_index.shape == (wl.N,)
    assert 10 * 20 <= wl.N <= 10 * 80
    ch = wl.children.reshape(-1, 4)
    arity = (ch >= 0).sum(1)
    assert arity.max() <= 4
    # slots are filled left to right
    for row in ch:
        k = int((row >= 0).sum())
        assert (row[:k] >= 0).all() and (row[k:] < 0).all()


def test_grid():
    wl = I.make_workload(4)
    assert (wl.N, wl.K, wl.H) == (65536, 2, 256)
    assert int((wl.children >= 0).sum()) == 126976
    assert wl.x.shape == (65536, 256) and wl.U.shape == (2, 256, 256)


def test_random_dag_is_acyclic_and_in_range():
    rng = np.random.default_rng(0)
    for _ in range(10):
        ch = I.random_dag(rng, 50, 3)
        assert ch.min() >= -1 and ch.max() < 50
