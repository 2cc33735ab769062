"""The paper's evaluation grid (TreeFC on perfect binary trees of height 7,
DAG-RNN on 10x10 grids, child-sum TreeLSTM and MV-RNN on SST-sized trees;
batch 1 and 10; hidden h_s and, where the library implements it, h_l):
every supported cell against the fp64 oracle, element by element, and the
unsupported hidden sizes rejected on the host."""
import numpy as np
import pytest

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import announce, compare_lin, compare_states, need_gpu

pytestmark = pytest.mark.gpu

SUPPORTED = [(c, b, "s") for c in I.PAPER_GRID_CELLS for b in (1, 10)] + \
            [(c, b, "l") for c in ("treefc", "dagrnn") for b in (1, 10)]
UNSUPPORTED = [("treegru", 1, "l"), ("treelstm", 1, "l"), ("mvrnn", 1, "l")]


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()


@pytest.mark.parametrize("cell,batch,hidden", SUPPORTED)
def test_paper_grid_parity(cell, batch, hidden):
    wl = I.paper_grid_workload(cell, batch, hidden)
    announce("paper grid %s batch %d h_%s (%s N=%d)" % (cell, batch, hidden, wl.name, wl.N))
    dw = DeviceWorkload(wl)
    dw.h.fill_(float("nan"))
    dw.step()
    assert dw.status_code() == 0
    compare_lin(dw.lin_host(), O.linearize(wl.children, wl.K), wl.K)
    compare_states(dw.states_by_node(), O.forward_workload(wl), wl.name)


@pytest.mark.parametrize("cell,batch,hidden", UNSUPPORTED)
def test_paper_grid_unsupported_hidden_rejected(cell, batch, hidden):
    wl = I.paper_grid_workload(cell, batch, hidden)
    announce("paper grid unsupported %s h_%s" % (cell, hidden))
    dw = DeviceWorkload(wl)
    dw.linearize()
    dw.h.fill_(7.0)
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0
    assert bool((dw.h == 7.0).all())          # nothing was enqueued
