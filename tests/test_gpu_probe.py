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
    assert C.cortex_probe_mfma(None, 10) == C.CORTEX_E_INVAL
    assert C.cortex_probe_mfma(sink, -1) == C.CORTEX_E_INVAL
