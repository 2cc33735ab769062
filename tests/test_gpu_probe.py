"""The matrix-core throughput probe: it launches, fills its sink with finite
values, reports the flop count its shape implies and rejects bad arguments."""
import pytest
import torch

from paper_2011_01383_amd import cortex as C
from tests.gpu_helpers import announce, need_gpu

pytestmark = pytest.mark.gpu


def test_probe_mfma():
    need_gpu()
    announce("probe mfma")
    n = C.cortex_probe_mfma_sink_floats()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert n == cus * 512
    assert C.cortex_probe_mfma_flops(10) == pytest.approx(cus * 8 * 10 * 16 * 2 * 16 * 16 * 4)
    sink = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    assert C.cortex_probe_mfma(sink, 10) == C.CORTEX_OK
    torch.cuda.synchronize()
    assert bool(torch.isfinite(sink).all())
    assert C.load().cortex_probe_mfma(None, 10, None) == C.CORTEX_E_INVAL
    with pytest.raises(ValueError, match="sink"):
        C.cortex_probe_mfma(None, 10)
    assert C.cortex_probe_mfma(sink, -1) == C.CORTEX_E_INVAL


@pytest.mark.parametrize("mode", [0, 1])
def test_probe_levels(mode):
    need_gpu()
    announce("probe levels mode %d" % mode)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ws = C.workspace(C.cortex_probe_levels_workspace_bytes())
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for grid, levels in ((cus, 0), (cus, 12), (7, 5), (1, 3), (cus, 12)):
        assert C.cortex_probe_levels(mode, grid, levels, status, ws) == C.CORTEX_OK
    torch.cuda.synchronize()
    assert int(status.item()) == 0


def test_probe_levels_rejects():
    need_gpu()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ws = C.workspace(C.cortex_probe_levels_workspace_bytes())
    small = C.workspace(256)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert C.cortex_probe_levels(2, cus, 4, status, ws) == C.CORTEX_E_INVAL
    assert C.cortex_probe_levels(0, 0, 4, status, ws) == C.CORTEX_E_INVAL
    assert C.cortex_probe_levels(0, cus, -1, status, ws) == C.CORTEX_E_INVAL
    assert C.cortex_probe_levels(0, cus + 1, 4, status, ws) == C.CORTEX_E_TOO_LARGE
    assert C.cortex_probe_levels(1, cus, 4, status, small) == C.CORTEX_E_WORKSPACE
    # a raised status ends the launch at once and is left as it was
    status.fill_(C.CORTEX_ST_CYCLE)
    assert C.cortex_probe_levels(1, cus, 4, status, ws) == C.CORTEX_OK
    torch.cuda.synchronize()
    assert int(status.item()) == C.CORTEX_ST_CYCLE
