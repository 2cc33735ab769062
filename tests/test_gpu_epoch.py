"""Launch tags come from the forward workspace, not from the host: every
forward launch that ends normally advances the workspace's staging epoch by
one (a sequence of per-level launches by one in all), two copies of the
library alternating on one workspace never reuse a tag, and a workspace whose
epoch has run out reports CORTEX_ST_EPOCH_WRAP, writes nothing and works
again once zeroed."""
import contextlib
import dataclasses
import shutil

import numpy as np
import pytest
import torch

from oracle import cortex_oracle as O
from paper_2011_01383_amd import cortex as C
from paper_2011_01383_amd import inputs as I
from paper_2011_01383_amd.runner import DeviceWorkload
from tests.gpu_helpers import announce, compare_states, need_gpu

pytestmark = pytest.mark.gpu

EPOCH_BYTE = 64          # word 16 of the workspace header


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()
    yield
    C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 0)
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, 0)


def epoch_of(ws):
    torch.cuda.synchronize()
    return int(ws[EPOCH_BYTE:EPOCH_BYTE + 4].view(torch.int32).item()) & 0xFFFFFFFF


CASES = {
    "nary_h256": (lambda: I.nary_treelstm_workload(91, batch=3, H=256), 0),
    "childsum_h256": (lambda: I.childsum_treelstm_workload(92, batch=3, H=256), 0),
    "treegru_h256": (lambda: I.childsum_treegru_workload(93, batch=3, H=256), 0),
    "mvrnn_d64": (lambda: I.mvrnn_workload(94, batch=3, d=64), 0),
    "dag_h256_units16": (lambda: I.dagrnn_workload(95, n_grids=2, rows=9, cols=7, H=256), 16),
    "dag_h256_units64": (lambda: I.dagrnn_workload(96, n_grids=2, rows=9, cols=7, H=256), 64),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_epoch_advances_once_per_forward(name):
    make, units = CASES[name]
    wl = make()
    announce("epoch advance %s N=%d" % (name, wl.N))
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, units)
    dw = DeviceWorkload(wl)
    dw.linearize()
    assert epoch_of(dw.ws_fwd) == 0
    ref = O.forward_workload(wl)
    for k in range(1, 4):
        dw.h.fill_(float("nan"))
        dw.forward()
        assert dw.status_code() == 0
        assert epoch_of(dw.ws_fwd) == k
        compare_states(dw.states_by_node(), ref, "%s launch %d" % (name, k))
    if name not in ("mvrnn_d64",):
        # one launch per level: one tag for the whole sequence
        C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 2)
        dw.h.fill_(float("nan"))
        dw.forward()
        assert dw.status_code() == 0
        assert epoch_of(dw.ws_fwd) == 4
        compare_states(dw.states_by_node(), ref, "%s per-level launches" % name)


@contextlib.contextmanager
def library(path):
    """Route the binding through another loaded copy of the library."""
    saved = C._lib
    C._lib = None
    try:
        C.load(path)
        yield
    finally:
        C._lib = saved


def test_two_library_copies_share_a_workspace(tmp_path):
    """A second copy of the library has its own host state; with host-side
    tag counters both copies would start from the same tag, and the second
    launch would take the first one's staged pairs for its own."""
    copy = str(tmp_path / "libcortex_copy.so")
    shutil.copyfile(C.LIB_PATH, copy)
    base = I.nary_treelstm_workload(97, batch=4, H=256)
    other = I.nary_treelstm_workload(98, batch=4, H=256)
    wl_b = dataclasses.replace(base, U=other.U, b=other.b)        # same trees, other weights
    announce("two library copies N=%d" % base.N)
    a = DeviceWorkload(base)
    b = DeviceWorkload(wl_b)
    b.ws_fwd = a.ws_fwd                                           # one workspace for both
    ref_a, ref_b = O.forward_workload(base), O.forward_workload(wl_b)
    assert np.abs(ref_a["h"] - ref_b["h"]).max() > 1e-2
    for rnd in range(3):
        for dw, ref, path in ((a, ref_a, None), (b, ref_b, copy)):
            ctx = library(path) if path else contextlib.nullcontext()
            with ctx:
                dw.h.fill_(float("nan"))
                dw.linearize()
                dw.forward()
                assert dw.status_code() == 0
            compare_states(dw.states_by_node(), ref, "round %d %s" % (rnd, "copy" if path else "main"))
    assert epoch_of(a.ws_fwd) == 6


def test_epoch_wrap_reports_and_recovers():
    wl = I.nary_treelstm_workload(99, batch=3, H=256)
    announce("epoch wrap N=%d" % wl.N)
    dw = DeviceWorkload(wl)
    dw.linearize()
    dw.ws_fwd[EPOCH_BYTE:EPOCH_BYTE + 4].view(torch.int32).fill_(-1)      # epoch 0xFFFFFFFF
    dw.h.fill_(7.0)
    dw.c.fill_(7.0)
    dw.forward()
    assert dw.status_code() == C.CORTEX_ST_EPOCH_WRAP
    assert bool((dw.h == 7.0).all()) and bool((dw.c == 7.0).all())
    dw.reset_status()                     # zeroes the status and the workspaces
    dw.step_two_calls()
    assert dw.status_code() == 0
    assert epoch_of(dw.ws_fwd) == 1
    compare_states(dw.states_by_node(), O.forward_workload(wl), "after zeroing")
