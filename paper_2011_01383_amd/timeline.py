"""Per-level timeline of one forward launch (trace build of the library).

    python -m paper_2011_01383_amd.timeline --workload 1 [--json out.json]

Loads ``libcortex_trace.so`` (built by ``python -m paper_2011_01383_amd.build
--trace``, i.e. with -DCORTEX_TRACE), runs a few warm passes of one workload,
clears the timeline, runs one more pass (the step's one launch where the
cell has a fused instance, else cortex_linearize then the forward;
``--two-calls`` forces the latter) and reads the stamps the forward kernel
left in its workspace: every workgroup (the first 256) stamps the
100 MHz wall clock at fixed points of every level.  The report gives, per
level, when the first workgroup entered it and when the last one left it
(both relative to the earliest kernel entry), the critical-path time of the
level (its last exit minus the previous level's last exit), and the longest
operand wait, contraction and epilogue of any workgroup's last tile there.

Stamp layout (uint64 ``trace[block][64][16]`` at byte offset
``SYNC_BYTES`` of the forward workspace): row ``l`` < 63 is level ``l``
(deeper levels share row 62); slot 0 level entry, 1 tile wait begins,
2 operands ready, 3 partial sums reduced, 4 tile written, 5 level exit,
6 first operands requested, 8 + w wave w finished its products.  Row 63
holds kernel-wide stamps: 0 entry, 1 weights resident, 2 structure ready,
3 exit.  Only the slice kernels (TreeRNN, N-ary and child-sum TreeLSTM,
DAG-RNN) stamp.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
TRACE_LIB = os.path.join(HERE, "libcortex_trace.so")

SYNC_BYTES = 128 + 4 * 4096 * 6          # workspace header (barrier, epoch and entered words) ahead of the timeline
TRACE_BLOCKS, TRACE_LEVELS, TRACE_SLOTS = 256, 64, 16
TICKS_PER_US = 100.0


def forward_ws(dw, fused):
    """The forward workspace of the last launch: the forward part of the
    cortex_tree_infer workspace for a fused launch, else the forward's own."""
    if not fused:
        return dw.ws_fwd
    from . import cortex as C
    lw = (C.cortex_linearize_workspace_bytes(dw.N, dw.K) + 255) // 256 * 256
    return dw.ws_inf[lw:]


def read_timeline(dw, fused=False):
    """The timeline of the last forward launch of ``dw`` as uint64 [256, 64, 16]."""
    import torch
    torch.cuda.synchronize()
    n = TRACE_BLOCKS * TRACE_LEVELS * TRACE_SLOTS * 8
    raw = forward_ws(dw, fused)[SYNC_BYTES:SYNC_BYTES + n].cpu().numpy()
    return raw.view(np.uint64).reshape(TRACE_BLOCKS, TRACE_LEVELS, TRACE_SLOTS)


def summarize(tr, num_levels, grid):
    """Per-level breakdown in microseconds from the raw stamps."""
    blocks = min(grid, TRACE_BLOCKS)
    tr = tr[:blocks].astype(np.int64)
    kern = tr[:, TRACE_LEVELS - 1, :]
    t0 = kern[:, 0][kern[:, 0] > 0].min()
    us = lambda t: float(t - t0) / TICKS_PER_US

    def span(a, b):
        """Largest b - a over blocks that stamped both."""
        m = (a > 0) & (b > 0)
        return float((b[m] - a[m]).max()) / TICKS_PER_US if m.any() else None

    out = {"kernel": {
        "entry_last_us": us(kern[:, 0][kern[:, 0] > 0].max()),
        "weights_resident_us": us(kern[:, 1].max()),
        "structure_ready_us": us(kern[:, 2].max()),
        "exit_us": us(kern[:, 3].max()),
    }, "levels": []}
    prev_exit = kern[:, 2].max()
    for l in range(min(num_levels, TRACE_LEVELS - 2)):
        row = tr[:, l, :]
        entered = row[:, 0][row[:, 0] > 0]
        exited = row[:, 5][row[:, 5] > 0]
        if entered.size == 0 or exited.size == 0:
            continue
        last_exit = exited.max()
        out["levels"].append({
            "level": l,
            "enter_first_us": us(entered.min()),
            "exit_last_us": us(last_exit),
            "critical_us": float(last_exit - prev_exit) / TICKS_PER_US,
            "wait_max_us": span(row[:, 1], row[:, 2]),
            "contract_max_us": span(row[:, 2], row[:, 3]),
            "epilogue_max_us": span(row[:, 3], row[:, 4]),
        })
        prev_exit = last_exit
    return out


def as_markdown(rep, title):
    k = rep["kernel"]
    lines = ["# Forward timeline: %s" % title, "",
             "Kernel: last entry %.2f us, weights resident %.2f us, structure ready %.2f us, exit %.2f us "
             "(all from the first workgroup's entry)." % (k["entry_last_us"], k["weights_resident_us"],
                                                          k["structure_ready_us"], k["exit_us"]), "",
             "| level | first entry (us) | last exit (us) | critical (us) | max wait (us) | max contraction (us) | max epilogue (us) |",
             "|---|---|---|---|---|---|---|"]
    f = lambda v: "-" if v is None else "%.2f" % v
    for r in rep["levels"]:
        lines.append("| %d | %s | %s | %s | %s | %s | %s |" % (
            r["level"], f(r["enter_first_us"]), f(r["exit_last_us"]), f(r["critical_us"]),
            f(r["wait_max_us"]), f(r["contract_max_us"]), f(r["epilogue_max_us"])))
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, default=1)
    ap.add_argument("--warm", type=int, default=5)
    ap.add_argument("--json", default=None)
    ap.add_argument("--markdown", default=None)
    ap.add_argument("--npy", default=None, help="also save the raw stamps, uint64 [256, 64, 16]")
    ap.add_argument("--lib", default=TRACE_LIB, help="trace build of the library to load")
    ap.add_argument("--two-calls", action="store_true",
                    help="trace cortex_linearize, then the forward entry point, instead of the step's launch")
    args = ap.parse_args()

    import torch
    from . import cortex as C
    from . import inputs as I
    from .runner import DeviceWorkload

    if not os.path.exists(args.lib):
        raise RuntimeError("%s is not built; run python -m paper_2011_01383_amd.build --trace" % args.lib)
    C.load(args.lib)
    torch.cuda.set_device(0)
    wl = I.make_workload(args.workload)
    dw = DeviceWorkload(wl)
    for _ in range(args.warm):
        dw.step()
    torch.cuda.synchronize()
    # a step is one launch where the batch's cell has a fused instance
    fused = C.cortex_last_grid(0) == 0 and not args.two_calls
    n = TRACE_BLOCKS * TRACE_LEVELS * TRACE_SLOTS * 8
    forward_ws(dw, fused)[SYNC_BYTES:SYNC_BYTES + n].zero_()
    dw.ws_lin.zero_()                     # a zeroed workspace is always a valid start
    if fused:
        dw.step()
        lin_stamps = np.zeros(7, dtype=np.int64)
    else:
        dw.linearize()
        torch.cuda.synchronize()
        lin_stamps = dw.ws_lin[:56].cpu().numpy().view(np.uint64).astype(np.int64)
        dw.forward()
    st = dw.status_code()
    if st != 0:
        raise RuntimeError("device status %d" % st)
    L = int(dw.lin_host()["num_levels"])
    raw = read_timeline(dw, fused)
    if args.npy:
        np.save(args.npy, raw)
    rep = summarize(raw, L, C.cortex_last_grid(1))
    rep["workload"] = wl.name
    rep["grid"] = C.cortex_last_grid(1)
    rep["num_levels"] = L
    lin_big = dw.ws_lin[:128].cpu().numpy().view(np.uint64).astype(np.int64)
    if C.cortex_last_grid(0) > 1 and lin_big[1] > 0:
        # multi-workgroup linearizer (workgroup 0's view): entry, heights,
        # histograms, scan, sort, offsets and child rows; height rounds and
        # the local sweeps of round 0
        t = lin_big[1:7]
        rep["linearize_big_phases_us"] = [float(x - t[0]) / TICKS_PER_US for x in t]
        rep["linearize_big_rounds"] = int(lin_big[7])
        rep["linearize_big_sweeps0"] = int(lin_big[8])
        # heights, round 0 (trace stamps 9-12 where present): children in
        # registers, dataflow pass done, local fixed point and heights written,
        # first grid barrier passed
        rep["linearize_big_round0_us"] = [float(x - t[0]) / TICKS_PER_US if x > 0 else None for x in lin_big[9:13]]
    if C.cortex_last_grid(0) == 1 and lin_stamps[0] > 0:
        # single-workgroup linearizer: entry, children loaded, heights done,
        # level counts, sort done, outputs written, offsets written
        rep["linearize_phases_us"] = [float(t - lin_stamps[0]) / TICKS_PER_US for t in lin_stamps]
    rep["one_launch"] = bool(fused)
    md = as_markdown(rep, "%s (grid %d, %d levels)" % (wl.name, rep["grid"], L))
    if fused:
        k0 = raw[0, TRACE_LEVELS - 1].astype(np.int64)
        lin = [float(k0[4 + i] - k0[4]) / TICKS_PER_US for i in range(5)] if k0[4] > 0 else None
        rep["linearize_in_kernel_us"] = lin
        md += ("\n\nOne launch: every workgroup linearizes the batch in LDS first, so \"weights resident\" and "
               "\"structure ready\" both mark the end of that linearization.")
        if lin:
            post = [float(k0[i] - k0[4]) / TICKS_PER_US if k0[i] > 0 else float("nan") for i in (9, 10)]
            rep["linearize_in_kernel_post_us"] = post
            md += (" Workgroup 0's linearizer, from its start: children loaded %.2f, heights %.2f, level counts and "
                   "offsets %.2f, sort %.2f us; linearization written out %.2f, structure cache built %.2f us."
                   % (tuple(lin[1:]) + tuple(post)))
    if "linearize_phases_us" in rep:
        md += ("\n\nLinearizer (one workgroup), from its entry: children loaded %.2f, heights %.2f, "
               "level counts and offsets %.2f, sort %.2f, outputs %.2f (end %.2f) us." % tuple(rep["linearize_phases_us"][1:]))
    if "linearize_big_phases_us" in rep:
        md += ("\n\nLinearizer (%d workgroups), workgroup 0 from its entry: heights %.2f (%d global rounds, "
               "%d local sweeps in round 0), histograms %.2f, scan %.2f, sort %.2f, offsets and child rows %.2f us."
               % (C.cortex_last_grid(0), rep["linearize_big_phases_us"][1], rep["linearize_big_rounds"],
                  rep["linearize_big_sweeps0"], *rep["linearize_big_phases_us"][2:]))
        r0 = rep["linearize_big_round0_us"]
        if all(v is not None for v in r0):
            md += (" Round 0 of the heights: children in registers %.2f, dataflow pass %.2f, local fixed point and "
                   "heights written %.2f, first grid barrier %.2f us." % tuple(r0))
    print(md)
    sys.stdout.flush()
    if args.json:
        with open(args.json, "w") as f:
            json.dump(rep, f, indent=1)
    if args.markdown:
        with open(args.markdown, "w") as f:
            f.write(md + "\n")


if __name__ == "__main__":
    main()
