"""Benchmark of the level-synchronous recursive-inference hot path on one GPU.

One step = one pass of the whole path over one batch: linearization (node
heights, level lists, child rows) and the persistent forward, through one
cortex_tree_infer / cortex_dag_infer call on one stream (a single launch where
the cell and batch have a fused instance) with the inputs already resident in
HBM.

Default workload: DAG-RNN, hidden 256, a batch of 64 image grids of 32 x 32
nodes (65,536 nodes, 63 anti-diagonal levels), the largest configuration; the
other four (TreeRNN H = 64 on one 32-leaf tree; binary N-ary TreeLSTM,
child-sum TreeLSTM and MV-RNN on batches of 10 random trees) are measured in
the same run under ``per_config``.

Prints ONE JSON line with the contract fields plus:
  roofline      the step's dominant kernel's achieved algorithmic FLOP/s (or
                GB/s) from its own HIP-event-timed launches, against the MI355X
                nominal peak and against the rate measured on the GPU itself
  cpu_baseline  the fp64 oracle on one host core: N over the median of 20
                passes (3 for the 65,536-node batch)
  breakdown     latency percentiles and the linearize / forward split
                (medians of single launches, averages of back-to-back ones)
  per_config    the same figures, condensed, for every other configuration
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "batch inference latency (ms) + nodes/sec; fraction of HBM/FLOP roofline"
PEAK_FP32_TFLOPS = 157.3        # MI355X dense fp32 (MFMA and vector)
PEAK_HBM_GBS = 8000.0           # MI355X HBM3E


def algorithmic_work(wl):
    """(flops, bytes) the method must do for one batch.

    Flops: 2 per multiply-add of the contractions actually needed (present
    child slots only, leaves of TreeRNN / N-ary / MV-RNN are copies) plus one
    per bias add.  Bytes: weights read once, inputs gathered once, every
    output state written once, the int32 structure read once.
    """
    H, K, N = wl.H, wl.K, wl.N
    ch = wl.children.reshape(N, K)
    present = ch >= 0
    E = int(present.sum())
    n_int = int(present.any(1).sum())
    n_leaf = N - n_int
    f4 = 4
    struct_bytes = N * K * 4 + N * 4
    if wl.cell == "tree_rnn":
        flops = E * 2 * H * H + n_int * H
        byts = (2 * H * H + H) * f4 + n_leaf * H * f4 + N * H * f4 + struct_bytes
    elif wl.cell == "nary_treelstm":
        flops = E * 2 * H * 5 * H + n_int * 5 * H
        byts = (2 * 5 * H * H + 5 * H) * f4 + n_leaf * H * f4 + 2 * N * H * f4 + struct_bytes
    elif wl.cell == "childsum_treelstm":
        flops = N * (2 * H * 4 * H + 4 * H) + n_int * 2 * H * 3 * H + E * 2 * H * H
        byts = (8 * H * H + 4 * H) * f4 + N * H * f4 + 2 * N * H * f4 + struct_bytes
    elif wl.cell in ("childsum_treegru", "simple_treegru"):
        # per node: W x for 3 gates + bias; per internal node: U_z h~, U_h m;
        # per child edge: U_r h_k
        flops = N * (2 * H * 3 * H + 3 * H) + n_int * 2 * (2 * H * H) + E * 2 * H * H
        byts = (6 * H * H + 3 * H) * f4 + N * H * f4 + N * H * f4 + struct_bytes
    elif wl.cell == "mvrnn":
        flops = n_int * (2 * H * 2 * H * H + 2 * 2 * H * H + 2 * H * 2 * H)
        byts = (2 * H * 2 * H) * f4 + n_leaf * (H * H + H) * f4 + N * (H * H + H) * f4 + struct_bytes
    else:  # dagrnn
        flops = N * (2 * H * H + H) + E * 2 * H * H
        byts = (3 * H * H + H) * f4 + N * H * f4 + N * H * f4 + struct_bytes
    return float(flops), float(byts)


def bound_of(flops, byts):
    """The roofline that bounds the algorithm: the larger ideal time wins."""
    t_f = flops / (PEAK_FP32_TFLOPS * 1e12)
    t_b = byts / (PEAK_HBM_GBS * 1e9)
    return "mfma" if t_f >= t_b else "hbm"


FORWARD_SOURCES = ("paper_2011_01383_amd/csrc/forward.hip", "paper_2011_01383_amd/csrc/cortex_device.hpp",
                   "paper_2011_01383_amd/csrc/cortex_host.hpp", "paper_2011_01383_amd/csrc/lin_small.hpp")


def forward_source_hash():
    """sha256 over the forward kernel's sources, to tell whether stored
    counter readings still describe the kernel that is built."""
    import hashlib
    h = hashlib.sha256()
    for rel in FORWARD_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(wl):
    """HBM bytes per forward launch from the rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary kept in profiles/ for this workload (each counter scaled by its
    reading on a plain copy of known size), or None when there is no summary
    or the forward sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "hbm_counters_%s.md" % wl.name)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.split(":", 1)[0].strip().isidentifier():
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha256") != forward_source_hash():
        return None
    try:
        return float(fields["forward_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def measured_peaks(stream):
    """Sustained rates of this GPU, beside the nominal peaks: fp32 matrix-core
    throughput from the library's register-only MFMA probe, and HBM bandwidth
    from a 1 GiB device copy (bytes read + bytes written).  Best of five
    launches each."""
    import torch
    from paper_2011_01383_amd import cortex as C

    def best_ms(fn, reps=5):
        fn()
        out = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b))
        return min(out)

    iters = 20000
    sink = torch.empty(C.cortex_probe_mfma_sink_floats(), dtype=torch.float32, device="cuda")
    C.check(C.cortex_probe_mfma(sink, 0, stream), "cortex_probe_mfma")
    mfma_ms = best_ms(lambda: C.cortex_probe_mfma(sink, iters, stream))
    n = (1 << 30) // 4
    src = torch.rand(n, device="cuda")
    dst = torch.empty_like(src)
    copy_ms = best_ms(lambda: dst.copy_(src))
    del src, dst
    return {"fp32_mfma_tflops": C.cortex_probe_mfma_flops(iters) / (mfma_ms / 1e3) / 1e12,
            "hbm_copy_gbs": 2.0 * n * 4 / (copy_ms / 1e3) / 1e9,
            "note": "register-only fp32 MFMA probe (16x16x4) on every CU; 1 GiB device copy, read + write"}


def level_floor(stream, grid, levels):
    """The fixed cost of a level loop at the forward's grid: an empty
    persistent launch, and per level the device-wide barrier (what a
    barrier-per-level schedule pays) and the per-datum all-to-all tagged
    exchange (what the forward's ordering pays at the least), each from
    cortex_probe_levels launched back to back with 0 and 64 empty levels."""
    import torch
    from paper_2011_01383_amd import cortex as C

    ws = C.workspace(C.cortex_probe_levels_workspace_bytes())
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    reps, deep = 50, 64

    def avg_us(mode, n_levels):
        run = lambda: C.check(C.cortex_probe_levels(mode, grid, n_levels, status, ws, stream), "cortex_probe_levels")
        for _ in range(5):
            run()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            run()
        b.record(stream)
        torch.cuda.synchronize()
        assert int(status.item()) == 0, "probe status %d" % int(status.item())
        return a.elapsed_time(b) * 1e3 / reps

    launch = avg_us(1, 0)
    barrier = (avg_us(0, deep) - launch) / deep
    exchange = (avg_us(1, deep) - launch) / deep
    return {"grid": grid, "levels": levels, "launch_us": launch, "barrier_us_per_level": barrier,
            "exchange_us_per_level": exchange, "barrier_floor_us": launch + (levels - 1) * barrier,
            "exchange_floor_us": launch + (levels - 1) * exchange,
            "note": "empty persistent launch + (levels - 1) x an empty level, 512-thread workgroups"}


def cpu_baseline(wl, runs):
    """The fp64 oracle (definitional linearization + recursive forward) timed
    pass by pass on one host thread; the value is N over the median pass."""
    from oracle import cortex_oracle as O
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=1)
    except Exception:          # threadpoolctl missing: BLAS may use more threads
        limiter = None
    lin_s, fwd_s = [], []
    for _ in range(runs):
        t0 = time.perf_counter()
        O.linearize(wl.children, wl.K)
        t1 = time.perf_counter()
        O.forward_workload(wl)
        t2 = time.perf_counter()
        lin_s.append(t1 - t0)
        fwd_s.append(t2 - t1)
    if limiter is not None:
        limiter.unregister()
    total = [a + b for a, b in zip(lin_s, fwd_s)]
    med = float(np.median(total))
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"value": wl.N / med, "unit": "nodes/s", "cores": 1, "kind": "oracle",
            "sample": "median of %d full passes over the %d-node batch (linearize + forward, fp64, 1 thread "
                      "of %s usable cores); %.1f s in all" % (runs, wl.N, affinity, sum(total)),
            "median_pass_s": med, "median_linearize_s": float(np.median(lin_s)),
            "median_forward_s": float(np.median(fwd_s))}


# Cortex's own latencies on the paper's V100 GPU, in ms (the GPU rows of the
# latency table comparing Cortex with DyNet, Sec. 7), keyed by (model,
# hidden size h_s / h_l, batch).  Context for the grid below, never a target:
# other hardware, and SST trees where the grid here uses SST-sized random ones.
PAPER_V100_CORTEX_MS = {
    ("treefc", "s", 1): 0.08, ("treefc", "s", 10): 0.17, ("treefc", "l", 1): 0.12, ("treefc", "l", 10): 0.37,
    ("dagrnn", "s", 1): 0.22, ("dagrnn", "s", 10): 0.39, ("dagrnn", "l", 1): 0.26, ("dagrnn", "l", 10): 0.54,
    ("treegru", "s", 1): 0.18, ("treegru", "s", 10): 0.35, ("treegru", "l", 1): 0.25, ("treegru", "l", 10): 0.75,
    ("treelstm", "s", 1): 0.24, ("treelstm", "s", 10): 0.39, ("treelstm", "l", 1): 0.29, ("treelstm", "l", 10): 0.70,
    ("mvrnn", "s", 1): 0.34, ("mvrnn", "s", 10): 0.78, ("mvrnn", "l", 1): 0.39, ("mvrnn", "l", 10): 1.11,
}


def paper_grid(args):
    """The paper's workload grid (models x batch {1, 10} x hidden {h_s, h_l});
    one JSON line per cell: step latency on this GPU (same protocol as the
    main bench), the roofline fraction of the step's forward kernel (the one
    launch of a step where linearization and forward are fused), and the
    paper's V100 latency as context.  Cells whose hidden size the library does not
    implement are reported as unsupported."""
    import torch
    from paper_2011_01383_amd import cortex as C
    from paper_2011_01383_amd import inputs as I
    from paper_2011_01383_amd.runner import DeviceWorkload
    stream = torch.cuda.current_stream()
    for cell in I.PAPER_GRID_CELLS:
        for hidden in ("s", "l"):
            for batch in (1, 10):
                wl = I.paper_grid_workload(cell, batch, hidden)
                line = {"grid_cell": cell, "hidden": wl.H, "hidden_class": "h_" + hidden, "batch": batch,
                        "workload": wl.name, "nodes": wl.N,
                        "paper_v100_cortex_ms": PAPER_V100_CORTEX_MS[(cell, hidden, batch)]}
                try:
                    dw = DeviceWorkload(wl)
                    dw.step()
                except RuntimeError as e:
                    line.update({"supported": False, "reason": str(e)})
                    print(json.dumps(line))
                    continue
                for _ in range(args.warmup):
                    dw.step()
                torch.cuda.synchronize()
                assert dw.status_code() == 0
                g0 = torch.cuda.Event(enable_timing=True)
                g1 = torch.cuda.Event(enable_timing=True)
                g0.record(stream)
                for _ in range(args.steps):
                    dw.step()
                g1.record(stream)
                torch.cuda.synchronize()
                assert dw.status_code() == 0
                ms = g0.elapsed_time(g1) / args.steps
                fused = C.cortex_last_grid(0) == 0
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                for _ in range(args.steps):
                    if fused:
                        dw.step()             # the one launch of a step
                    else:
                        dw.forward()
                b.record(stream)
                torch.cuda.synchronize()
                fwd_ms = a.elapsed_time(b) / args.steps
                flops, byts = algorithmic_work(wl)
                bound = bound_of(flops, byts)
                frac = (flops / (fwd_ms / 1e3) / 1e12 / PEAK_FP32_TFLOPS if bound == "mfma"
                        else byts / (fwd_ms / 1e3) / 1e9 / PEAK_HBM_GBS)
                line.update({"supported": True, "levels": int(dw.lin_host()["num_levels"]), "ms_per_step": ms,
                             "nodes_per_s": wl.N / (ms / 1e3), "forward_ms": fwd_ms, "one_launch": fused,
                             "bound": bound, "roofline_frac": frac})
                print(json.dumps(line))
                sys.stdout.flush()


def ablation(args):
    """How the forward orders its levels (CORTEX_KNOB_LEVEL_SYNC): per-datum
    waits in one persistent launch (the default), plus a device-wide barrier
    after every level, or one launch per level that reloads weights and
    structure each time; for the TreeGRU cells also a barrier after each of
    the level's two exchanges (the schedule without recursive refactoring,
    Secs. 3.1 and 7.4); for the 64-grid DAG-RNN also the input products
    hoisted into one matrix product before the level loop (ABLATE bit 2)
    instead of fused into each tile.  Then, on the N-ary TreeLSTM and TreeFC
    batches, the optimizations of Sec. 7.3 switched off (CORTEX_KNOB_ABLATE):
    model persistence, leaf specialization, both, and both with one launch
    per level.  One JSON line per (workload, mode): the forward kernel time (for
    mode 2, the whole per-level launch sequence, which also synchronizes once
    to read L), the median of five rounds in which every schedule of a
    workload is timed once."""
    import torch
    from paper_2011_01383_amd import cortex as C
    from paper_2011_01383_amd import inputs as I
    from paper_2011_01383_amd.runner import DeviceWorkload
    stream = torch.cuda.current_stream()
    names = {0: "per-datum waits, one launch", 1: "plus a device-wide barrier per level",
             2: "one launch per level",
             3: "a device-wide barrier after each of the two exchanges per level"}
    cases = [(I.make_workload(1), 0), (I.make_workload(2), 0),
             (I.childsum_treegru_workload(I.BASE_SEED + 60, batch=10, H=256), 0),
             (I.childsum_treegru_workload(I.BASE_SEED + 60, batch=10, H=256, simple=True), 0),
             (I.make_workload(4), 64)]
    runs = []
    for wl, units in cases:
        for mode in ((0, 1, 3, 2) if wl.cell in (I.CELL_CHILDSUM_TREEGRU, I.CELL_SIMPLE_TREEGRU) else (0, 1, 2)):
            runs.append((wl, units, mode, 0))
        if wl.cell == I.CELL_DAGRNN:
            # the input products hoisted into one matrix product ahead of the
            # level loop (Sec. 7.1), against the fused input part
            runs.append((wl, units, 0, 4))
    # optimizations switched off one at a time, then all with one launch per
    # level (Sec. 7.3): model persistence (bit 0), leaf specialization (bit 1)
    for wl in (I.make_workload(1), I.treefc_workload(I.BASE_SEED + 61, batch=10, H=256)):
        for mode, bits in ((0, 0), (0, 1), (0, 2), (0, 3), (2, 3)):
            runs.append((wl, 0, mode, bits))
    abl_names = {0: "", 1: "; weights read from memory at every tile", 2: "; leaf states staged and waited for",
                 3: "; weights from memory and leaf states staged",
                 4: "; input products hoisted into one matrix product before the level loop"}
    def knobs(units, mode, bits):
        C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, units)
        C.cortex_set_knob(C.CORTEX_KNOB_LEVEL_SYNC, mode)
        C.cortex_set_knob(C.CORTEX_KNOB_ABLATE, bits)

    n = max(10, min(args.steps, 100))
    rounds = 5
    groups = []                           # runs of one workload, timed interleaved
    for run in runs:
        if groups and groups[-1][0][0] is run[0]:
            groups[-1].append(run)
        else:
            groups.append([run])
    for group in groups:
        live = []
        for wl, units, mode, bits in group:
            knobs(units, mode, bits)
            line = {"workload": wl.name, "level_sync": mode, "ablate": bits, "mode": names[mode] + abl_names[bits]}
            dw = DeviceWorkload(wl)
            dw.linearize()
            try:
                dw.forward()
            except RuntimeError as e:
                line.update({"supported": False, "reason": str(e)})
                live.append((line, None, (units, mode, bits), []))
                continue
            line["grid"] = C.cortex_last_grid(1)
            for _ in range(args.warmup):
                dw.forward()
            torch.cuda.synchronize()
            assert dw.status_code() == 0
            live.append((line, dw, (units, mode, bits), []))
        # every schedule of the workload timed once per round, so slow drifts
        # of the machine touch them alike; the median of the rounds is reported
        for _ in range(rounds):
            for line, dw, kb, times in live:
                if dw is None:
                    continue
                knobs(*kb)
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                for _ in range(n):
                    dw.forward()
                b.record(stream)
                torch.cuda.synchronize()
                assert dw.status_code() == 0
                times.append(a.elapsed_time(b) / n)
        for line, dw, kb, times in live:
            if dw is not None:
                line.update({"supported": True, "forward_ms": float(np.median(times)), "forward_ms_min": min(times),
                             "forward_ms_rounds": times, "levels": int(dw.lin_host()["num_levels"])})
            print(json.dumps(line))
            sys.stdout.flush()
        knobs(0, 0, 0)


def unroll_study(args):
    """Unrolled recursion for TreeRNN at H = 64 (Secs. 3.1, 7.4;
    CORTEX_KNOB_TREE_UNROLL): the whole batch in one workgroup (up to 320
    nodes), one workgroup per tree, and level-parallel hidden slices that
    exchange states between workgroups at every level.  One JSON line per
    (batch, schedule): the forward kernel time and the step as the two calls
    (cortex_linearize, then cortex_tree_forward, so that every schedule is
    timed the same way), both averaged over back-to-back launches between two
    events."""
    import torch
    from paper_2011_01383_amd import cortex as C
    from paper_2011_01383_amd import inputs as I
    from paper_2011_01383_amd.runner import DeviceWorkload
    stream = torch.cuda.current_stream()
    names = {0: "whole batch in one workgroup", 1: "level-parallel hidden slices", 2: "one workgroup per tree"}
    cases = [I.make_workload(0), I.tree_rnn_forest_workload(I.BASE_SEED + 80, batch=5),
             I.tree_rnn_forest_workload(I.BASE_SEED + 81, batch=10),
             I.tree_rnn_forest_workload(I.BASE_SEED + 82, batch=32, leaf_lo=10, leaf_hi=40),
             I.tree_rnn_forest_workload(I.BASE_SEED + 83, batch=100, leaf_lo=2, leaf_hi=18)]
    n = max(10, min(args.steps, 100))

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    for wl in cases:
        for mode in (0, 2, 1):
            if mode == 0 and wl.N > 320:
                continue
            C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, mode)
            dw = DeviceWorkload(wl)
            dw.step()
            torch.cuda.synchronize()
            assert dw.status_code() == 0
            fwd = timed(dw.forward)
            step = timed(dw.step_two_calls)
            assert dw.status_code() == 0
            print(json.dumps({"workload": wl.name, "nodes": wl.N, "levels": int(dw.lin_host()["num_levels"]),
                              "schedule": names[mode], "tree_unroll": mode, "grid": C.cortex_last_grid(1),
                              "forward_ms": fwd, "step_ms": step}))
            sys.stdout.flush()
        C.cortex_set_knob(C.CORTEX_KNOB_TREE_UNROLL, 0)


def dag_batches(args):
    """DAG-RNN at H = 256 over growing batches of 32 x 32 grids (the paper's
    DAG-RNN cell, Sec. 7.1; 16 to 512 grids, 16,384 to 524,288 nodes, all 63
    levels): the forward kernel and the step (cortex_dag_infer: linearizer,
    then forward), each averaged over back-to-back launches between two
    events (the median of three rounds), and the forward's algorithmic rate
    against the fp32 peak.  One JSON line per batch.  Larger batches give each node group more steps
    per level, so the per-level exchange is spread over more work."""
    import torch
    from paper_2011_01383_amd import inputs as I
    from paper_2011_01383_amd.runner import DeviceWorkload
    stream = torch.cuda.current_stream()
    n = max(5, min(args.steps, 50))

    def timed(fn):
        # the median of three rounds of n launches each
        for _ in range(max(args.warmup, 5)):
            fn()
        torch.cuda.synchronize()
        rounds = []
        for _ in range(3):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(n):
                fn()
            b.record(stream)
            torch.cuda.synchronize()
            rounds.append(a.elapsed_time(b) / n)
        return sorted(rounds)[1]

    for grids in (16, 32, 64, 128, 256, 512):
        wl = I.dagrnn_workload(I.BASE_SEED + 2000 + grids, n_grids=grids)
        dw = DeviceWorkload(wl)
        dw.step()
        torch.cuda.synchronize()
        assert dw.status_code() == 0
        fwd = timed(dw.forward)
        step = timed(dw.step)
        assert dw.status_code() == 0
        flops, _ = algorithmic_work(wl)
        print(json.dumps({"workload": wl.name, "grids": grids, "nodes": wl.N, "levels": int(dw.lin_host()["num_levels"]),
                          "forward_ms": fwd, "step_ms": step, "nodes_per_s": wl.N / (step * 1e-3),
                          "forward_tflops": flops / (fwd * 1e-3) * 1e-12,
                          "forward_frac": flops / (fwd * 1e-3) * 1e-12 / PEAK_FP32_TFLOPS}))
        sys.stdout.flush()
        del dw
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=4,
                    help="headline configuration 0..4: tree_rnn, nary, childsum, mvrnn, dag (default: the "
                         "64-grid DAG-RNN batch, the largest)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="measure the headline configuration only (no per_config entries)")
    ap.add_argument("--node-groups", type=int, default=0)
    ap.add_argument("--slice-units", type=int, default=0, help="hidden units per forward slice (0 = default)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB mebibytes (reads MIB, writes MIB) "
                         "five times, to scale HBM byte counters; prints one JSON line")
    ap.add_argument("--paper-grid", action="store_true",
                    help="run the paper's model x batch x hidden-size grid; one JSON line per cell")
    ap.add_argument("--ablation", action="store_true",
                    help="forward time under each level-ordering mode; one JSON line per (workload, mode)")
    ap.add_argument("--unroll", action="store_true",
                    help="TreeRNN H = 64 batches under each unrolling schedule; one JSON line per (batch, schedule)")
    ap.add_argument("--dag-batches", action="store_true",
                    help="DAG-RNN H = 256 over 16 to 512 grids of 32x32; one JSON line per batch")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the path shards by whole trees/grids with no "
              "exchange, and this implementation has no multi-GPU run", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.rand(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_mib": args.calibrate_copy, "launches": 5,
                          "bytes_read_per_launch": n * 4, "bytes_written_per_launch": n * 4}))
        return
    from paper_2011_01383_amd import cortex as C
    from paper_2011_01383_amd import inputs as I
    from paper_2011_01383_amd.runner import DeviceWorkload

    if not os.path.exists(C.LIB_PATH):
        from paper_2011_01383_amd import build
        build.build()
    torch.cuda.set_device(0)
    if args.paper_grid:
        paper_grid(args)
        return
    if args.ablation:
        ablation(args)
        return
    if args.unroll:
        unroll_study(args)
        return
    if args.dag_batches:
        dag_batches(args)
        return
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_NODE_GROUPS, args.node_groups)
    C.cortex_set_knob(C.CORTEX_KNOB_FWD_SLICE_UNITS, args.slice_units)
    stream = torch.cuda.current_stream()
    peaks = measured_peaks(stream)
    wl = I.make_workload(args.workload)
    head = measure(wl, args, stream, peaks, full=True)
    others = []
    if not args.no_other_configs:
        for k in range(len(I.WORKLOADS)):
            if k != args.workload:
                others.append(measure(I.make_workload(k), args, stream, peaks, full=False))

    out = {
        "metric": METRIC,
        "value": head["nodes_per_s"],
        "unit": "nodes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded)",
        "config": head["config"],
        "roofline": head["roofline"],
        "cpu_baseline": head["cpu_baseline"],
        "level_floor": head["level_floor"],
        "breakdown": head["breakdown"],
        "per_config": others,
    }
    print(json.dumps(out))


def measure(wl, args, stream, peaks, full):
    """One configuration: K steps between two events (value = N / ms_per_step),
    per-step latencies, the step's launches and the two separate calls timed
    launch by launch (medians) and back to back (averages, as a kernel trace
    reports them), the dominant kernel's roofline fraction and the oracle on
    one host core.  full=False keeps the fields a per-configuration summary
    needs."""
    import torch
    from paper_2011_01383_amd import cortex as C
    from paper_2011_01383_amd.runner import DeviceWorkload

    dw = DeviceWorkload(wl)
    for _ in range(args.warmup):
        dw.step()
    torch.cuda.synchronize()
    assert dw.status_code() == 0, "device status %d" % dw.status_code()

    # ---- timed region: exactly K steps, events only at its two ends (an
    #      event between steps is a GPU command of its own and would add its
    #      cost to every step) ----
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g0 = torch.cuda.Event(enable_timing=True)
    g1 = torch.cuda.Event(enable_timing=True)
    g0.record(stream)
    for _ in range(args.steps):
        dw.step()
    g1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = g0.elapsed_time(g1)
    assert dw.status_code() == 0
    ms_per_step = total_ms / args.steps

    def per_launch_ms(fn, n):
        """n calls, each between its own event pair (includes the events' cost)."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        fn()
        torch.cuda.synchronize()
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev])

    def back_to_back_ms(fn, n):
        """Average duration of n calls between two events on the launch stream."""
        for _ in range(5):            # host-side first-call work stays out of the average
            fn()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    step_ms = per_launch_ms(dw.step, args.steps)
    n_k = max(20, min(args.steps, 200))
    # the step's own launch(es): one cortex_tree_infer / cortex_dag_infer
    # call, a single fused kernel where the cell and batch have one (the
    # linearizer grid is then reported as 0); the two-call components are
    # timed beside it
    step_avg_ms = back_to_back_ms(dw.step, n_k)
    grid_lin, grid_fwd = C.cortex_last_grid(0), C.cortex_last_grid(1)
    fused = grid_lin == 0
    lin_avg_ms = back_to_back_ms(dw.linearize, n_k)
    fwd_avg_ms = back_to_back_ms(dw.forward, n_k)
    lin_ms = per_launch_ms(dw.linearize, n_k)
    fwd_ms = per_launch_ms(dw.forward, n_k)
    assert dw.status_code() == 0

    flops, byts = algorithmic_work(wl)
    bound = bound_of(flops, byts)
    kern_ms = step_avg_ms if fused else fwd_avg_ms

    def frac_at(ms):
        if bound == "mfma":
            return flops / (ms / 1e3) / 1e12 / PEAK_FP32_TFLOPS
        return byts / (ms / 1e3) / 1e9 / PEAK_HBM_GBS

    if bound == "mfma":
        achieved = flops / (kern_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_FP32_TFLOPS}
        roof["peak_measured"] = peaks["fp32_mfma_tflops"]
    else:
        achieved = byts / (kern_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
        roof["peak_measured"] = peaks["hbm_copy_gbs"]
    roof["traffic"] = measured_traffic(wl)
    roof["frac_of_measured"] = achieved / roof["peak_measured"]
    roof["peak_measured_note"] = peaks["note"]
    roof["traffic_unit"] = "bytes per launch"
    roof["traffic_source"] = ("profiles/hbm_counters_%s.md: rocprofv3 FETCH_SIZE and WRITE_SIZE passes, each scaled "
                              "by its reading on a plain copy; used only while the forward sources hash as they did "
                              "when the counters were taken (null otherwise)" % wl.name)
    roof["kernel"] = ("linearize + forward in one launch (%s)" if fused else "forward (%s)") % wl.cell
    roof["kernel_avg_ms"] = kern_ms
    roof["algorithmic_flops"] = flops
    roof["algorithmic_bytes"] = byts

    lin_host = dw.lin_host()
    levels = int(lin_host["num_levels"])
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, 3 if wl.N > 20000 else 20)
    config = {"workload": wl.name, "cell": wl.cell, "hidden": wl.H, "nodes": wl.N, "levels": levels,
              "max_arity": wl.K, "grid_linearize": grid_lin, "grid_forward": grid_fwd, "one_launch": fused}
    res = {"config": config, "ms_per_step": ms_per_step, "nodes_per_s": wl.N / (ms_per_step / 1e3),
           "latency_ms_p50": float(np.percentile(step_ms, 50)), "roofline": roof, "cpu_baseline": cpu}
    if not full:
        res["roofline"] = {k: roof[k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic", "kernel",
                                                "kernel_avg_ms")}
        res["linearize_ms_median"] = float(np.median(lin_ms))
        res["forward_ms_median"] = float(np.median(fwd_ms))
        return res
    res["level_floor"] = level_floor(stream, grid_fwd, levels)
    res["breakdown"] = {
        "latency_note": "percentiles from a second pass with an event pair around each step (includes the "
                        "events' own cost)",
        "latency_ms_p10": float(np.percentile(step_ms, 10)),
        "latency_ms_p50": float(np.percentile(step_ms, 50)),
        "latency_ms_p90": float(np.percentile(step_ms, 90)),
        "nodes_per_s_at_p50": wl.N / (float(np.percentile(step_ms, 50)) / 1e3),
        "step_launches_avg_ms": step_avg_ms,
        "two_calls_note": "cortex_linearize and cortex_tree_forward / cortex_dag_forward on their own: medians "
                          "of launches each between its own event pair, and averages of back-to-back launches",
        "linearize_ms_median": float(np.median(lin_ms)),
        "forward_ms_median": float(np.median(fwd_ms)),
        "linearize_kernel_avg_ms": lin_avg_ms,
        "forward_kernel_avg_ms": fwd_avg_ms,
        "roofline_frac_forward_only": frac_at(fwd_avg_ms),
        "roofline_frac_end_to_end": frac_at(ms_per_step),
        "measured_fp32_mfma_tflops": peaks["fp32_mfma_tflops"],
        "measured_hbm_copy_gbs": peaks["hbm_copy_gbs"],
        "host_wall_s": wall,
    }
    return res


if __name__ == "__main__":
    main()
