"""C-ABI checks that need no GPU: the library loads, exports every function
declared in include/cortex.h, and rejects bad arguments on the host before
enqueuing anything."""
import ctypes
import os
import re

import pytest

from paper_2011_01383_amd import cortex as C

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cortex.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(cortex_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(C.LIB_PATH):
        from paper_2011_01383_amd import build
        build.build()
    return C.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("cortex_linearize", "cortex_tree_forward", "cortex_dag_forward",
                     "cortex_linearize_workspace_bytes", "cortex_forward_workspace_bytes"):
        assert required in names
    assert sorted(C.EXPORTED) == names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version(lib):
    assert "gfx950" in C.cortex_version()


def test_workspace_sizes(lib):
    assert C.cortex_linearize_workspace_bytes(10, 5) == 0          # K out of range
    assert C.cortex_linearize_workspace_bytes(-1, 2) == 0
    small = C.cortex_linearize_workspace_bytes(100, 2)
    big = C.cortex_linearize_workspace_bytes(100000, 2)
    assert 0 < small < big
    assert big >= 2 * 100000 * 4                                  # two permutation buffers
    assert C.cortex_forward_workspace_bytes(1, 368, 256) > 0
    assert C.cortex_forward_workspace_bytes(9, 368, 256) == 0


def test_host_validation_returns_before_any_device_work(lib):
    lin = C.cortex_lin_t(10, 2, None, None, None, None, None, None)
    # K out of range, N mismatch, NULL status: all rejected on the host
    assert lib.cortex_linearize(None, 10, 5, ctypes.byref(lin), None, None, 0, None) == C.CORTEX_E_INVAL
    assert lib.cortex_linearize(None, 11, 2, ctypes.byref(lin), ctypes.c_void_p(8), None, 0, None) == C.CORTEX_E_INVAL
    assert lib.cortex_linearize(None, 10, 2, None, ctypes.c_void_p(8), None, 0, None) == C.CORTEX_E_INVAL
    w = C.cortex_weights_t(None, None, None, None)
    assert lib.cortex_tree_forward(7, 256, ctypes.byref(lin), None, 0, None, None, ctypes.byref(w),
                                   None, None, ctypes.c_void_p(8), None, 0, None) == C.CORTEX_E_INVAL
    assert lib.cortex_dag_forward(256, None, None, None, None, None, None, None, None, 0, None) == C.CORTEX_E_INVAL


def test_knobs(lib):
    old = C.cortex_get_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS)
    assert C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, 3) == C.CORTEX_OK
    assert C.cortex_get_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS) == 3
    assert C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, old) == C.CORTEX_OK
    assert C.cortex_set_knob(99, 1) == C.CORTEX_E_INVAL
    assert C.cortex_set_knob(C.CORTEX_KNOB_LIN_BLOCKS, -1) == C.CORTEX_E_INVAL
    assert C.cortex_get_knob(C.CORTEX_KNOB_BARRIER_TIMEOUT_US) > 0


def test_level_sync_knob_range(lib):
    assert C.cortex_get_knob(C.CORTEX_KNOB_LEVEL_SYNC) == 0
    assert C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, 4) == C.CORTEX_E_INVAL
    for v in (3, 2, 1, 0):
        assert C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, v) == C.CORTEX_OK
        assert C.cortex_get_knob(C.CORTEX_KNOB_LEVEL_SYNC) == v
    assert C.cortex_set_knob(C.CORTEX_KNOB_ABLATE + 1, 0) == C.CORTEX_E_INVAL


def test_ablate_knob_range(lib):
    assert C.cortex_get_knob(C.CORTEX_KNOB_ABLATE) == 0
    assert C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, 8) == C.CORTEX_E_INVAL
    for v in (7, 6, 5, 4, 3, 2, 1, 0):
        assert C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, v) == C.CORTEX_OK
        assert C.cortex_get_knob(C.CORTEX_KNOB_ABLATE) == v


def test_tree_unroll_knob_range(lib):
    assert C.cortex_get_knob(C.CORTEX_KNOB_TREE_UNROLL) == 0
    assert C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 3) == C.CORTEX_E_INVAL
    for v in (2, 1, 0):
        assert C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, v) == C.CORTEX_OK
        assert C.cortex_get_knob(C.CORTEX_KNOB_TREE_UNROLL) == v


# ---- the binding rejects tensors the library would misread (no GPU needed) ----

def _cpu(n, dtype):
    import torch
    return torch.zeros(n, dtype=dtype)


def test_binding_rejects_wrong_dtype_before_the_call():
    import torch
    # an int64 children array would be read as int32 pairs: a different tree
    with pytest.raises(ValueError, match="children must be torch.int32"):
        C.cortex_linearize(_cpu(20, torch.int64), 10, 2, None, None, None)
    with pytest.raises(ValueError, match="x must be torch.float32"):
        C._check_dag_args(256, 4, _cpu(4 * 256, torch.float16), None, None, None, None, None, None)


def test_binding_rejects_short_and_strided_tensors():
    import torch
    with pytest.raises(ValueError, match="children holds 19 elements, needs at least 20"):
        C.cortex_linearize(_cpu(19, torch.int32), 10, 2, None, None, None)
    strided = torch.zeros(40, dtype=torch.int32)[::2]
    with pytest.raises(ValueError, match="children must be contiguous"):
        C.cortex_linearize(strided, 10, 2, None, None, None)
    with pytest.raises(ValueError, match="N must be non-negative"):
        C.cortex_linearize(_cpu(4, torch.int32), -2, 2, None, None, None)


def test_binding_rejects_host_memory():
    import torch
    with pytest.raises(ValueError, match="children must be in device memory"):
        C.cortex_linearize(_cpu(20, torch.int32), 10, 2, None, None, None)
    with pytest.raises(ValueError, match="num_levels must be in device memory"):
        C.Linearization.alloc(10, 2, device="cpu")


def test_binding_checks_weight_and_table_sizes():
    import torch
    H, N = 64, 5
    f32 = torch.float32
    idx = _cpu(N, torch.int32)
    # x_rows larger than the table: the buffer descriptor would cover memory past it
    with pytest.raises(ValueError, match="x_table holds 640 elements, needs at least 704"):
        C._check_tree_args(C.CORTEX_TREE_RNN, H, N, _cpu(10 * H, f32), 11, idx, None,
                           {"W": _cpu(2 * H * H, f32), "b": _cpu(H, f32)}, _cpu(N * H, f32), None, None, None)
    # an N-ary U holding one child's gates only
    with pytest.raises(ValueError, match="U holds"):
        C._check_tree_args(C.CORTEX_NARY_TREELSTM, H, N, _cpu(10 * H, f32), 10, idx, None,
                           {"U": _cpu(5 * H * H, f32), "b": _cpu(5 * H, f32)}, _cpu(N * H, f32),
                           _cpu(N * H, f32), None, None)
    # MV-RNN: P must hold N matrices
    with pytest.raises(ValueError, match="P holds"):
        C._check_tree_args(C.CORTEX_MVRNN, H, N, _cpu(10 * H, f32), 10, idx, _cpu(10 * H * H, f32),
                           {"W": _cpu(2 * H * H, f32), "W_M": _cpu(2 * H * H, f32)}, _cpu(N * H, f32),
                           _cpu(N * H, f32), None, None)
    # all sizes right: the first complaint is that the memory is on the host
    with pytest.raises(ValueError, match="x_table must be in device memory"):
        C._check_tree_args(C.CORTEX_TREE_RNN, H, N, _cpu(10 * H, f32), 10, idx, None,
                           {"W": _cpu(2 * H * H, f32), "b": _cpu(H, f32)}, _cpu(N * H, f32), None,
                           _cpu(1, torch.int32), _cpu(256, torch.uint8))
