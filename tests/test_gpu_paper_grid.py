"""The paper's evaluation grid (TreeFC on perfect binary trees of height 7,
DAG-RNN on 10x10 grids, child-sum TreeLSTM and MV-RNN on SST-sized trees;
batch 1 and 10; hidden h_s and h_l): every cell against the fp64 oracle,
element by element, and hidden sizes without a kernel instance rejected on
the host."""
import numpy as np
import pytest

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import announce, compare_lin, compare_states, need_gpu

pytestmark = pytest.mark.gpu

SUPPORTED = [(c, b, h) for c in I.PAPER_GRID_CELLS for b in (1, 10) for h in ("s", "l")]


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


@pytest.mark.parametrize("maker", [
    lambda: I.childsum_treelstm_workload(5, batch=1, H=128),
    lambda: I.childsum_treegru_workload(5, batch=1, H=1024),
    lambda: I.mvrnn_workload(5, batch=1, d=96),
])
def test_unsupported_hidden_rejected(maker):
    """A hidden size no kernel instance exists for is refused on the host."""
    wl = maker()
    announce("unsupported hidden %s H=%d" % (wl.cell, wl.H))
    dw = DeviceWorkload(wl)
    dw.linearize()
    dw.h.fill_(7.0)
    with pytest.raises(RuntimeError, match="host code %d" % C.CORTEX_E_INVAL):
        dw.forward()
    assert dw.status_code() == 0
    assert bool((dw.h == 7.0).all())          # nothing was enqueued
