"""ctypes binding of libcortex.so (the C ABI in include/cortex.h).

The functions below carry the C names and only marshal arguments: every step
of linearization and of the forward pass runs in the library's HIP kernels.
PyTorch serves as the allocator of device memory and the source of streams.
Loading fails loudly when the library has not been built; there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcortex.so")

CORTEX_OK = 0
CORTEX_E_INVAL = -1
CORTEX_E_HIP = -2
CORTEX_E_TOO_LARGE = -3
CORTEX_E_WORKSPACE = -4

CORTEX_ST_OK = 0
CORTEX_ST_CHILD_RANGE = 1
CORTEX_ST_CYCLE = 2
CORTEX_ST_BARRIER_TIMEOUT = 3
CORTEX_ST_BAD_LINEARIZATION = 4
CORTEX_ST_INPUT_RANGE = 5

CORTEX_TREE_RNN = 0
CORTEX_NARY_TREELSTM = 1
CORTEX_CHILDSUM_TREELSTM = 2
CORTEX_MVRNN = 3
CORTEX_CHILDSUM_TREEGRU = 4
CORTEX_SIMPLE_TREEGRU = 5

CORTEX_KNOB_LIN_BLOCKS = 0
CORTEX_KNOB_FWD_NODE_GROUPS = 1
CORTEX_KNOB_BARRIER_TIMEOUT_US = 2
CORTEX_KNOB_COOPERATIVE = 3
CORTEX_KNOB_FWD_SLICE_UNITS = 4
CORTEX_KNOB_LEVEL_SYNC = 5
CORTEX_KNOB_TREE_UNROLL = 6
CORTEX_KNOB_ABLATE = 7

CELL_IDS = {"tree_rnn": CORTEX_TREE_RNN, "nary_treelstm": CORTEX_NARY_TREELSTM,
            "childsum_treelstm": CORTEX_CHILDSUM_TREELSTM, "mvrnn": CORTEX_MVRNN,
            "childsum_treegru": CORTEX_CHILDSUM_TREEGRU, "simple_treegru": CORTEX_SIMPLE_TREEGRU}

EXPORTED = [
    "cortex_linearize_workspace_bytes", "cortex_linearize", "cortex_forward_workspace_bytes",
    "cortex_tree_forward", "cortex_dag_forward", "cortex_tree_infer_workspace_bytes", "cortex_tree_infer",
    "cortex_dag_infer_workspace_bytes", "cortex_dag_infer",
    "cortex_set_knob", "cortex_get_knob",
    "cortex_last_grid", "cortex_version",
    "cortex_probe_mfma_sink_floats", "cortex_probe_mfma_flops", "cortex_probe_mfma",
    "cortex_probe_levels_workspace_bytes", "cortex_probe_levels",
]


class cortex_lin_t(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("max_arity", ctypes.c_int32),
                ("num_levels", ctypes.c_void_p), ("height", ctypes.c_void_p),
                ("level_offsets", ctypes.c_void_p), ("level_nodes", ctypes.c_void_p),
                ("node_row", ctypes.c_void_p), ("child_rows", ctypes.c_void_p)]


class cortex_weights_t(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("U", ctypes.c_void_p), ("b", ctypes.c_void_p),
                ("W_M", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libcortex.so and declare the signatures (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libcortex.so is not built (%s); run paper_2011_01383_amd.build" % path)
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.cortex_linearize_workspace_bytes.argtypes = [I32, I32]
    lib.cortex_linearize_workspace_bytes.restype = SZ
    lib.cortex_linearize.argtypes = [P, I32, I32, ctypes.POINTER(cortex_lin_t), P, P, SZ, P]
    lib.cortex_linearize.restype = ctypes.c_int
    lib.cortex_forward_workspace_bytes.argtypes = [I32, I32, I32]
    lib.cortex_forward_workspace_bytes.restype = SZ
    lib.cortex_tree_forward.argtypes = [I32, I32, ctypes.POINTER(cortex_lin_t), P, I32, P, P,
                                        ctypes.POINTER(cortex_weights_t), P, P, P, P, SZ, P]
    lib.cortex_tree_forward.restype = ctypes.c_int
    lib.cortex_dag_forward.argtypes = [I32, ctypes.POINTER(cortex_lin_t), P, P, P, P, P, P, P, SZ, P]
    lib.cortex_dag_forward.restype = ctypes.c_int
    lib.cortex_tree_infer_workspace_bytes.argtypes = [I32, I32, I32, I32]
    lib.cortex_tree_infer_workspace_bytes.restype = SZ
    lib.cortex_tree_infer.argtypes = [I32, I32, P, ctypes.POINTER(cortex_lin_t), P, I32, P, P,
                                      ctypes.POINTER(cortex_weights_t), P, P, P, P, SZ, P]
    lib.cortex_tree_infer.restype = ctypes.c_int
    lib.cortex_dag_infer_workspace_bytes.argtypes = [I32, I32, I32]
    lib.cortex_dag_infer_workspace_bytes.restype = SZ
    lib.cortex_dag_infer.argtypes = [I32, P, ctypes.POINTER(cortex_lin_t), P, P, P, P, P, P, P, SZ, P]
    lib.cortex_dag_infer.restype = ctypes.c_int
    lib.cortex_set_knob.argtypes = [I32, I64]
    lib.cortex_set_knob.restype = ctypes.c_int
    lib.cortex_get_knob.argtypes = [I32]
    lib.cortex_get_knob.restype = I64
    lib.cortex_last_grid.argtypes = [I32]
    lib.cortex_last_grid.restype = I32
    lib.cortex_probe_mfma_sink_floats.argtypes = []
    lib.cortex_probe_mfma_sink_floats.restype = SZ
    lib.cortex_probe_mfma_flops.argtypes = [I32]
    lib.cortex_probe_mfma_flops.restype = ctypes.c_double
    lib.cortex_probe_mfma.argtypes = [P, I32, P]
    lib.cortex_probe_mfma.restype = ctypes.c_int
    lib.cortex_probe_levels_workspace_bytes.argtypes = []
    lib.cortex_probe_levels_workspace_bytes.restype = SZ
    lib.cortex_probe_levels.argtypes = [I32, I32, I32, P, P, SZ, P]
    lib.cortex_probe_levels.restype = ctypes.c_int
    lib.cortex_version.argtypes = []
    lib.cortex_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ---- the C entry points, same names -------------------------------------------

def cortex_linearize_workspace_bytes(N: int, K: int) -> int:
    return load().cortex_linearize_workspace_bytes(N, K)


def cortex_forward_workspace_bytes(cell: int, N: int, H: int) -> int:
    return load().cortex_forward_workspace_bytes(cell, N, H)


def cortex_linearize(children: torch.Tensor, N: int, K: int, lin: "Linearization",
                     status: torch.Tensor, ws: torch.Tensor, stream=None) -> int:
    return load().cortex_linearize(_ptr(children), N, K, ctypes.byref(lin.struct), _ptr(status),
                                   _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))


def cortex_tree_forward(cell: int, H: int, lin: "Linearization", x_table: Optional[torch.Tensor],
                        x_rows: int, x_index: torch.Tensor, leaf_mat: Optional[torch.Tensor],
                        W=None, U=None, b=None, W_M=None, h: torch.Tensor = None,
                        c_or_P: Optional[torch.Tensor] = None, status: torch.Tensor = None,
                        ws: torch.Tensor = None, stream=None) -> int:
    w = cortex_weights_t(_ptr(W), _ptr(U), _ptr(b), _ptr(W_M))
    return load().cortex_tree_forward(cell, H, ctypes.byref(lin.struct), _ptr(x_table), x_rows,
                                      _ptr(x_index), _ptr(leaf_mat), ctypes.byref(w), _ptr(h),
                                      _ptr(c_or_P), _ptr(status), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream(stream))


def cortex_dag_forward(H: int, lin: "Linearization", x: torch.Tensor, W: torch.Tensor,
                       U: torch.Tensor, b: torch.Tensor, h: torch.Tensor, status: torch.Tensor,
                       ws: torch.Tensor, stream=None) -> int:
    return load().cortex_dag_forward(H, ctypes.byref(lin.struct), _ptr(x), _ptr(W), _ptr(U), _ptr(b),
                                     _ptr(h), _ptr(status), _ptr(ws), ws.numel() * ws.element_size(),
                                     _stream(stream))


def cortex_tree_infer_workspace_bytes(cell: int, N: int, K: int, H: int) -> int:
    return load().cortex_tree_infer_workspace_bytes(cell, N, K, H)


def cortex_tree_infer(cell: int, H: int, children: torch.Tensor, lin: "Linearization",
                      x_table: Optional[torch.Tensor], x_rows: int, x_index: torch.Tensor,
                      leaf_mat: Optional[torch.Tensor], W=None, U=None, b=None, W_M=None,
                      h: torch.Tensor = None, c_or_P: Optional[torch.Tensor] = None,
                      status: torch.Tensor = None, ws: torch.Tensor = None, stream=None) -> int:
    w = cortex_weights_t(_ptr(W), _ptr(U), _ptr(b), _ptr(W_M))
    return load().cortex_tree_infer(cell, H, _ptr(children), ctypes.byref(lin.struct), _ptr(x_table), x_rows,
                                    _ptr(x_index), _ptr(leaf_mat), ctypes.byref(w), _ptr(h), _ptr(c_or_P),
                                    _ptr(status), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))


def cortex_dag_infer_workspace_bytes(N: int, K: int, H: int) -> int:
    return load().cortex_dag_infer_workspace_bytes(N, K, H)


def cortex_dag_infer(H: int, children: torch.Tensor, lin: "Linearization", x: torch.Tensor, W: torch.Tensor,
                     U: torch.Tensor, b: torch.Tensor, h: torch.Tensor, status: torch.Tensor, ws: torch.Tensor,
                     stream=None) -> int:
    return load().cortex_dag_infer(H, _ptr(children), ctypes.byref(lin.struct), _ptr(x), _ptr(W), _ptr(U),
                                   _ptr(b), _ptr(h), _ptr(status), _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream(stream))


def cortex_set_knob(knob: int, value: int) -> int:
    return load().cortex_set_knob(knob, value)


def cortex_get_knob(knob: int) -> int:
    return load().cortex_get_knob(knob)


def cortex_last_grid(which: int) -> int:
    return load().cortex_last_grid(which)


def cortex_probe_mfma_sink_floats() -> int:
    return load().cortex_probe_mfma_sink_floats()


def cortex_probe_mfma_flops(iters: int) -> float:
    return load().cortex_probe_mfma_flops(iters)


def cortex_probe_mfma(sink: torch.Tensor, iters: int, stream=None) -> int:
    return load().cortex_probe_mfma(_ptr(sink), iters, _stream(stream))


def cortex_probe_levels_workspace_bytes() -> int:
    return load().cortex_probe_levels_workspace_bytes()


def cortex_probe_levels(mode: int, grid: int, levels: int, status: torch.Tensor, ws: torch.Tensor,
                        stream=None) -> int:
    return load().cortex_probe_levels(mode, grid, levels, _ptr(status), _ptr(ws), ws.numel() * ws.element_size(),
                                      _stream(stream))


def cortex_version() -> str:
    return load().cortex_version().decode()


# ---- device-memory plumbing ---------------------------------------------------

@dataclass
class Linearization:
    """Caller-owned device arrays of a linearization (cortex_lin_t)."""
    N: int
    K: int
    num_levels: torch.Tensor
    height: torch.Tensor
    level_offsets: torch.Tensor
    level_nodes: torch.Tensor
    node_row: torch.Tensor
    child_rows: torch.Tensor

    def __post_init__(self):
        self.struct = cortex_lin_t(self.N, self.K, _ptr(self.num_levels), _ptr(self.height),
                                   _ptr(self.level_offsets), _ptr(self.level_nodes),
                                   _ptr(self.node_row), _ptr(self.child_rows))

    @staticmethod
    def alloc(N: int, K: int, device="cuda") -> "Linearization":
        e = lambda n: torch.empty(max(n, 1), dtype=torch.int32, device=device)
        return Linearization(N, K, e(1), e(N), e(N + 1), e(N), e(N), e(N * K))


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """Zero-filled workspace (the library requires zeros before first use)."""
    return torch.zeros(max(1, (nbytes + 255) // 256 * 256), dtype=torch.uint8, device=device)


def check(rc: int, what: str = "cortex call") -> None:
    if rc != CORTEX_OK:
        raise RuntimeError("%s failed with host code %d" % (what, rc))
