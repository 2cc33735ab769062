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
CORTEX_ST_EPOCH_WRAP = 6

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
    "cortex_tree_infer_noalloc",
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
    lib.cortex_tree_infer_noalloc.argtypes = [I32, I32, P, ctypes.POINTER(cortex_lin_t), P, I32, P, P,
                                              ctypes.POINTER(cortex_weights_t), P, P, P, P]
    lib.cortex_tree_infer_noalloc.restype = ctypes.c_int
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


def _need(t, name: str, dtype: torch.dtype, min_numel: int, optional: bool = False) -> None:
    """Reject a tensor the library would misread: the library takes raw
    pointers, so a wrong dtype, a strided view, too few elements or host
    memory would be read as something else (or past the allocation)."""
    _need_all([(t, name, dtype, min_numel, optional)])


def _need_all(specs) -> None:
    """_need over several tensors: every dtype, layout and size first, then
    that each tensor is in device memory."""
    for t, name, dtype, min_numel, optional in specs:
        if t is None:
            if optional:
                continue
            raise ValueError("%s is required" % name)
        if not isinstance(t, torch.Tensor):
            raise ValueError("%s must be a torch.Tensor, got %s" % (name, type(t).__name__))
        if dtype is not None and t.dtype != dtype:
            raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous" % name)
        if t.numel() < min_numel:
            raise ValueError("%s holds %d elements, needs at least %d" % (name, t.numel(), min_numel))
    for t, name, _, _, _ in specs:
        if t is not None and not t.is_cuda:
            raise ValueError("%s must be in device memory" % name)


def _need_count(v: int, name: str) -> None:
    if int(v) < 0:
        raise ValueError("%s must be non-negative, got %d" % (name, int(v)))


# Elements of each weight tensor per cell, as functions of H (layouts of the
# header: row-major [out, in] float32).
_WEIGHT_ELEMS = {
    CORTEX_TREE_RNN: {"W": lambda H: 2 * H * H, "b": lambda H: H},
    CORTEX_NARY_TREELSTM: {"U": lambda H: 10 * H * H, "b": lambda H: 5 * H},
    CORTEX_CHILDSUM_TREELSTM: {"W": lambda H: 4 * H * H, "U": lambda H: 4 * H * H, "b": lambda H: 4 * H},
    CORTEX_MVRNN: {"W": lambda H: 2 * H * H, "W_M": lambda H: 2 * H * H},
    CORTEX_CHILDSUM_TREEGRU: {"W": lambda H: 3 * H * H, "U": lambda H: 3 * H * H, "b": lambda H: 3 * H},
    CORTEX_SIMPLE_TREEGRU: {"W": lambda H: 3 * H * H, "U": lambda H: 3 * H * H, "b": lambda H: 3 * H},
}


_NO_WS = object()        # the entry point takes no workspace


def _check_tree_args(cell: int, H: int, N: int, x_table, x_rows: int, x_index, leaf_mat, weights: dict, h,
                     c_or_P, status, ws) -> None:
    if cell not in _WEIGHT_ELEMS:
        return                      # the library rejects the cell id itself
    _need_count(H, "H")
    _need_count(x_rows, "x_rows")
    f32, i32 = torch.float32, torch.int32
    specs = [(x_table, "x_table", f32, x_rows * H, x_rows == 0), (x_index, "x_index", i32, N, False)]
    if cell == CORTEX_MVRNN:
        specs.append((leaf_mat, "leaf_mat", f32, x_rows * H * H, x_rows == 0))
    for name, elems in _WEIGHT_ELEMS[cell].items():
        specs.append((weights.get(name), name, f32, elems(H), False))
    specs.append((h, "h", f32, N * H, False))
    if cell in (CORTEX_NARY_TREELSTM, CORTEX_CHILDSUM_TREELSTM):
        specs.append((c_or_P, "c", f32, N * H, False))
    elif cell == CORTEX_MVRNN:
        specs.append((c_or_P, "P", f32, N * H * H, False))
    specs.append((status, "status", i32, 1, False))
    if ws is not _NO_WS:
        specs.append((ws, "ws", None, 1, False))
    _need_all(specs)


def _check_dag_args(H: int, N: int, x, W, U, b, h, status, ws) -> None:
    _need_count(H, "H")
    f32 = torch.float32
    _need_all([(x, "x", f32, N * H, False), (W, "W", f32, H * H, False), (U, "U", f32, 2 * H * H, False),
               (b, "b", f32, H, False), (h, "h", f32, N * H, False), (status, "status", torch.int32, 1, False),
               (ws, "ws", None, 1, False)])


def _check_lin(lin: "Linearization", N: int, K: int) -> None:
    if not isinstance(lin, Linearization):
        raise ValueError("lin must be a Linearization")
    if lin.N != N or lin.K != K:
        raise ValueError("lin was allocated for N=%d K=%d, the call has N=%d K=%d" % (lin.N, lin.K, N, K))


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
    _need_count(N, "N")
    _need_count(K, "K")
    _need(children, "children", torch.int32, N * K)
    _check_lin(lin, N, K)
    _need(status, "status", torch.int32, 1)
    _need(ws, "ws", None, 1)
    return load().cortex_linearize(_ptr(children), N, K, ctypes.byref(lin.struct), _ptr(status),
                                   _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))


def cortex_tree_forward(cell: int, H: int, lin: "Linearization", x_table: Optional[torch.Tensor],
                        x_rows: int, x_index: torch.Tensor, leaf_mat: Optional[torch.Tensor],
                        W=None, U=None, b=None, W_M=None, h: torch.Tensor = None,
                        c_or_P: Optional[torch.Tensor] = None, status: torch.Tensor = None,
                        ws: torch.Tensor = None, stream=None) -> int:
    _check_lin(lin, lin.N, lin.K)
    _check_tree_args(cell, H, lin.N, x_table, x_rows, x_index, leaf_mat, {"W": W, "U": U, "b": b, "W_M": W_M},
                     h, c_or_P, status, ws)
    w = cortex_weights_t(_ptr(W), _ptr(U), _ptr(b), _ptr(W_M))
    return load().cortex_tree_forward(cell, H, ctypes.byref(lin.struct), _ptr(x_table), x_rows,
                                      _ptr(x_index), _ptr(leaf_mat), ctypes.byref(w), _ptr(h),
                                      _ptr(c_or_P), _ptr(status), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream(stream))


def cortex_dag_forward(H: int, lin: "Linearization", x: torch.Tensor, W: torch.Tensor,
                       U: torch.Tensor, b: torch.Tensor, h: torch.Tensor, status: torch.Tensor,
                       ws: torch.Tensor, stream=None) -> int:
    _check_lin(lin, lin.N, lin.K)
    _check_dag_args(H, lin.N, x, W, U, b, h, status, ws)
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
    _check_lin(lin, lin.N, lin.K)
    _need(children, "children", torch.int32, lin.N * lin.K)
    _check_tree_args(cell, H, lin.N, x_table, x_rows, x_index, leaf_mat, {"W": W, "U": U, "b": b, "W_M": W_M},
                     h, c_or_P, status, ws)
    w = cortex_weights_t(_ptr(W), _ptr(U), _ptr(b), _ptr(W_M))
    return load().cortex_tree_infer(cell, H, _ptr(children), ctypes.byref(lin.struct), _ptr(x_table), x_rows,
                                    _ptr(x_index), _ptr(leaf_mat), ctypes.byref(w), _ptr(h), _ptr(c_or_P),
                                    _ptr(status), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))


def cortex_tree_infer_noalloc(cell: int, H: int, children: torch.Tensor, lin: "Linearization",
                              x_table: Optional[torch.Tensor], x_rows: int, x_index: torch.Tensor,
                              leaf_mat: Optional[torch.Tensor], W=None, U=None, b=None, W_M=None,
                              h: torch.Tensor = None, c_or_P: Optional[torch.Tensor] = None,
                              status: torch.Tensor = None, stream=None) -> int:
    _check_lin(lin, lin.N, lin.K)
    _need(children, "children", torch.int32, lin.N * lin.K)
    _check_tree_args(cell, H, lin.N, x_table, x_rows, x_index, leaf_mat, {"W": W, "U": U, "b": b, "W_M": W_M},
                     h, c_or_P, status, _NO_WS)
    w = cortex_weights_t(_ptr(W), _ptr(U), _ptr(b), _ptr(W_M))
    return load().cortex_tree_infer_noalloc(cell, H, _ptr(children), ctypes.byref(lin.struct), _ptr(x_table), x_rows,
                                            _ptr(x_index), _ptr(leaf_mat), ctypes.byref(w), _ptr(h), _ptr(c_or_P),
                                            _ptr(status), _stream(stream))


def cortex_dag_infer_workspace_bytes(N: int, K: int, H: int) -> int:
    return load().cortex_dag_infer_workspace_bytes(N, K, H)


def cortex_dag_infer(H: int, children: torch.Tensor, lin: "Linearization", x: torch.Tensor, W: torch.Tensor,
                     U: torch.Tensor, b: torch.Tensor, h: torch.Tensor, status: torch.Tensor, ws: torch.Tensor,
                     stream=None) -> int:
    _check_lin(lin, lin.N, lin.K)
    _need(children, "children", torch.int32, lin.N * lin.K)
    _check_dag_args(H, lin.N, x, W, U, b, h, status, ws)
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
    _need(sink, "sink", torch.float32, cortex_probe_mfma_sink_floats())
    return load().cortex_probe_mfma(_ptr(sink), iters, _stream(stream))


def cortex_probe_levels_workspace_bytes() -> int:
    return load().cortex_probe_levels_workspace_bytes()


def cortex_probe_levels(mode: int, grid: int, levels: int, status: torch.Tensor, ws: torch.Tensor,
                        stream=None) -> int:
    _need(status, "status", torch.int32, 1)
    _need(ws, "ws", None, 1)
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
        sizes = {"num_levels": 1, "height": self.N, "level_offsets": self.N + 1, "level_nodes": self.N,
                 "node_row": self.N, "child_rows": self.N * self.K}
        for name, n in sizes.items():
            _need(getattr(self, name), name, torch.int32, n)
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
