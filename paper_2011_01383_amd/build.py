"""Builds libcortex.so (gfx950) in-tree with hipcc.

    python -m paper_2011_01383_amd.build

Every HIP source under csrc/ is compiled for gfx950 with packed-FP32 code
generation disabled, then linked into ``paper_2011_01383_amd/libcortex.so``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcortex.so")
TRACE_LIB = os.path.join(HERE, "libcortex_trace.so")
ARCH = os.environ.get("CORTEX_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "-O3", "--offload-arch=" + ARCH, "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]
SOURCES = ["abi.hip", "linearize.hip", "forward.hip", "probe.hip"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def build(verbose: bool = False, trace: bool = False) -> str:
    """Compile every source and link the shared library; returns its path.

    ``trace=True`` builds libcortex_trace.so with -DCORTEX_TRACE (per-level
    timeline stamps in the forward workspace) beside the regular library.
    """
    hipcc = _hipcc()
    build_dir = BUILD + ("_trace" if trace else "")
    lib = TRACE_LIB if trace else LIB
    os.makedirs(build_dir, exist_ok=True)
    extra = ["-DCORTEX_TRACE"] if trace else []

    def compile_one(src: str) -> str:
        obj = os.path.join(build_dir, src.replace(".hip", ".o"))
        cmd = [hipcc, *HIPCC_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed on %s:\n%s" % (src, r.stderr))
        if verbose:
            print(" ".join(cmd))
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = lib + ".tmp"
    cmd = [hipcc, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s" % r.stderr)
    os.replace(tmp, lib)
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv, trace="--trace" in sys.argv)
