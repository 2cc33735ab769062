"""Host-side logic of bench.py (no GPU): the algorithmic work of the 64-grid
DAG-RNN batch against its closed form, the roofline each workload is bound
by, the hash gate on stored HBM counters, and the one-GPU guard."""
import os
import subprocess
import sys

import pytest

import bench
from paper_2011_01383_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_dag_grid_work_closed_form():
    # 64 grids of 32 x 32: every node runs W x (a 256 x 256 matrix-vector
    # product) plus its bias; each of the 64 * 2 * 32 * 31 child edges one
    # more product with U_up or U_left.  Bytes: x and h of every node, the
    # three weight matrices and the bias once, children and one word per node.
    wl = I.make_workload(4)
    flops, byts = bench.algorithmic_work(wl)
    n, h = 64 * 32 * 32, 256
    edges = 64 * 2 * 32 * 31
    assert wl.N == n
    assert flops == pytest.approx(8.590e9 + 16.643e9 + n * h, rel=1e-3)
    assert flops == n * (2 * h * h + h) + edges * 2 * h * h
    assert byts == pytest.approx(2 * n * h * 4 + 3 * h * h * 4 + h * 4 + n * 3 * 4, rel=1e-12)


@pytest.mark.parametrize("k,bound", [(0, "hbm"), (1, "mfma"), (2, "mfma"), (3, "mfma"), (4, "mfma")])
def test_bounds(k, bound):
    # the 32-leaf TreeRNN moves more bytes than its few flops take at the
    # fp32 rate; every other workload is bound by the matrix cores
    assert bench.bound_of(*bench.algorithmic_work(I.make_workload(k))) == bound


def test_stored_traffic_needs_matching_sources(monkeypatch):
    wl = I.make_workload(4)
    monkeypatch.setattr(bench, "forward_source_hash", lambda: "0" * 64)
    assert bench.measured_traffic(wl) is None


def test_stored_traffic_read_when_sources_match(monkeypatch):
    # a summary is read exactly when its recorded source hash is the current one
    for k in range(5):
        wl = I.make_workload(k)
        with open(os.path.join(ROOT, "profiles", "hbm_counters_%s.md" % wl.name)) as f:
            stored = [ln.split(":", 1)[1].strip() for ln in f if ln.startswith("kernel_source_sha256:")]
        assert len(stored) == 1
        monkeypatch.setattr(bench, "forward_source_hash", lambda: stored[0])
        t = bench.measured_traffic(wl)
        assert t is not None and t > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
