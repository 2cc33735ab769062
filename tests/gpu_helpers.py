"""Shared helpers of the GPU parity tests (imported by tests/test_gpu_*.py)."""
import functools
import sys

import numpy as np
import pytest

ATOL_MAX = 1e-4     # max |gpu - oracle| per state tensor
ATOL_MEAN = 1e-5    # mean |gpu - oracle| per state tensor


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2011_01383_amd import cortex as C
    C.load()          # raises if the library is missing: no silent fallback


def announce(msg):
    """Name the case before its GPU step (survives a box that dies)."""
    print("[gpu-case]", msg, flush=True)
    sys.stdout.flush()


def compare_lin(got, ref, K):
    assert int(got["num_levels"]) == int(ref["num_levels"])
    for key in ("height", "level_offsets", "level_nodes", "node_row", "child_rows"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)


def compare_states(got, ref, label=""):
    for key, r in ref.items():
        g = got[key]
        assert g.shape == r.shape, (key, g.shape, r.shape)
        assert np.isfinite(g).all(), "%s %s has non-finite values" % (label, key)
        d = np.abs(g - r)
        mx, mean = float(d.max()), float(d.mean())
        assert mx <= ATOL_MAX, "%s %s max|d| = %.3g" % (label, key, mx)
        assert mean <= ATOL_MEAN, "%s %s mean|d| = %.3g" % (label, key, mean)


@functools.lru_cache(maxsize=None)
def cached_workload(k, j):
    from paper_2011_01383_amd import inputs as I
    return I.make_workload(k, j)


@functools.lru_cache(maxsize=None)
def cached_oracle(k, j):
    from oracle import cortex_oracle as O
    return O.forward_workload(cached_workload(k, j))


@functools.lru_cache(maxsize=None)
def cached_oracle_lin(k, j):
    from oracle import cortex_oracle as O
    wl = cached_workload(k, j)
    return O.linearize(wl.children, wl.K)
