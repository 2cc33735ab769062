"""Device-side driver of the hot path for one workload.

``DeviceWorkload`` uploads a workload's structure, inputs and weights once,
allocates the caller-owned linearization, outputs, status word and workspaces,
and enqueues the path on one stream through ``cortex_tree_infer`` or
``cortex_dag_infer`` (linearization and forward in one call, one launch where
the cell and batch have a fused instance); the two separate entry points can
also be called on their own.  It only marshals
arguments; all the work is done by the library's kernels.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import cortex as C


class DeviceWorkload:
    def __init__(self, wl, device: str = "cuda", stream=None):
        C.load()
        self.wl = wl
        self.device = device
        self.stream = stream
        dev = lambda a, dt=None: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.N, self.K, self.H = wl.N, wl.K, wl.H
        self.children = dev(wl.children)
        self.x_index = dev(wl.x_index)
        self.x_table = dev(wl.x_table)
        self.leaf_mat = dev(wl.leaf_mat)
        self.x = dev(wl.x)
        self.W, self.U, self.b, self.W_M = dev(wl.W), dev(wl.U), dev(wl.b), dev(wl.W_M)
        self.lin = C.Linearization.alloc(self.N, self.K, device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.ws_lin = C.workspace(C.cortex_linearize_workspace_bytes(self.N, self.K), device)
        self.is_dag = wl.cell == "dagrnn"
        self.cell = -1 if self.is_dag else C.CELL_IDS[wl.cell]
        self.ws_fwd = C.workspace(C.cortex_forward_workspace_bytes(self.cell, self.N, self.H), device)
        self.ws_inf = C.workspace(C.cortex_dag_infer_workspace_bytes(self.N, self.K, self.H) if self.is_dag else
                                  C.cortex_tree_infer_workspace_bytes(self.cell, self.N, self.K, self.H), device)
        rows = max(self.N, 1)
        self.h = torch.empty(rows, self.H, dtype=torch.float32, device=device)
        if wl.cell in ("nary_treelstm", "childsum_treelstm"):
            self.c = torch.empty(rows, self.H, dtype=torch.float32, device=device)
        elif wl.cell == "mvrnn":
            self.c = torch.empty(rows, self.H, self.H, dtype=torch.float32, device=device)
        else:
            self.c = None
        self.x_rows = 0 if wl.x_table is None else int(wl.x_table.shape[0])

    # ---- the two entry points ------------------------------------------------
    def linearize(self) -> None:
        C.check(C.cortex_linearize(self.children, self.N, self.K, self.lin, self.status, self.ws_lin,
                                   self.stream), "cortex_linearize")

    def forward(self) -> None:
        if self.is_dag:
            rc = C.cortex_dag_forward(self.H, self.lin, self.x, self.W, self.U, self.b, self.h,
                                      self.status, self.ws_fwd, self.stream)
        else:
            rc = C.cortex_tree_forward(self.cell, self.H, self.lin, self.x_table, self.x_rows,
                                       self.x_index, self.leaf_mat, W=self.W, U=self.U, b=self.b,
                                       W_M=self.W_M, h=self.h, c_or_P=self.c, status=self.status,
                                       ws=self.ws_fwd, stream=self.stream)
        C.check(rc, "forward")

    def infer(self) -> None:
        """Linearization and forward in one call (cortex_tree_infer or cortex_dag_infer)."""
        if self.is_dag:
            rc = C.cortex_dag_infer(self.H, self.children, self.lin, self.x, self.W, self.U, self.b, self.h,
                                    self.status, self.ws_inf, self.stream)
        else:
            rc = C.cortex_tree_infer(self.cell, self.H, self.children, self.lin, self.x_table, self.x_rows,
                                     self.x_index, self.leaf_mat, W=self.W, U=self.U, b=self.b, W_M=self.W_M,
                                     h=self.h, c_or_P=self.c, status=self.status, ws=self.ws_inf,
                                     stream=self.stream)
        C.check(rc, "infer")

    def step(self) -> None:
        """One pass of the hot path: linearization and forward through the
        one-call entry point (one launch where the cell and batch allow)."""
        self.infer()

    def step_two_calls(self) -> None:
        """The same pass as cortex_linearize, then the forward entry point."""
        self.linearize()
        self.forward()

    # ---- results -------------------------------------------------------------
    def status_code(self) -> int:
        torch.cuda.synchronize()
        return int(self.status.item())

    def reset_status(self) -> None:
        """Clear the status word and, as the ABI requires after an error, the workspaces."""
        self.status.zero_()
        self.ws_lin.zero_()
        self.ws_fwd.zero_()
        self.ws_inf.zero_()

    def lin_host(self) -> Dict[str, np.ndarray]:
        torch.cuda.synchronize()
        L = int(self.lin.num_levels.item())
        N, K = self.N, self.K
        return {
            "num_levels": np.int32(L),
            "height": self.lin.height[:N].cpu().numpy(),
            "level_offsets": self.lin.level_offsets[:L + 1].cpu().numpy(),
            "level_nodes": self.lin.level_nodes[:N].cpu().numpy(),
            "node_row": self.lin.node_row[:N].cpu().numpy(),
            "child_rows": self.lin.child_rows[:N * K].cpu().numpy(),
        }

    def states_by_node(self) -> Dict[str, np.ndarray]:
        """Outputs permuted from row order back to node-id order."""
        torch.cuda.synchronize()
        node_row = self.lin.node_row[:self.N].long()
        out = {"h": self.h[node_row].double().cpu().numpy()}
        if self.c is not None:
            out["P" if self.wl.cell == "mvrnn" else "c"] = self.c[node_row].double().cpu().numpy()
        return out
