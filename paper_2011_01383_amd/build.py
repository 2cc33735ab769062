"""Builds libcortex.so (gfx950) in-tree with hipcc.

    python -m paper_2011_01383_amd.build

Every HIP source under csrc/ is compiled for gfx950 with packed-FP32 code
generation disabled, then linked into ``paper_2011_01383_amd/libcortex.so``.

The feature flag reaches both of hipcc's passes; the host (x86) pass does not
know it and warns, the gfx950 pass honours it.  The build does not rely on the
flag alone: it disassembles the gfx950 code object of every source it just
compiled and fails if any packed-FP32 arithmetic instruction is present.
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
SOURCES = ["abi.hip", "linearize.hip", "forward.hip", "probe.hip", "noalloc.hip"]
# packed two-lane fp32 arithmetic, which this library must not contain
PACKED_FP32 = ("v_pk_add_f32", "v_pk_mul_f32", "v_pk_fma_f32")
LLVM_BIN = "/opt/rocm/llvm/bin"


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _llvm_tool(name: str) -> str:
    for cand in (os.path.join(LLVM_BIN, name), shutil.which(name)):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("%s not found: the device code cannot be checked" % name)


def check_no_packed_fp32(obj: str) -> int:
    """Disassemble the gfx950 code object embedded in one compiled object file
    and raise if it holds a packed-FP32 arithmetic instruction.  Returns the
    number of instructions checked (0 for a host-only object)."""
    sections = subprocess.run([_llvm_tool("llvm-readelf"), "-S", obj], capture_output=True, text=True, check=True)
    if ".hip_fatbin" not in sections.stdout:
        return 0
    fatbin, dev = obj + ".fatbin", obj + ".gfx.o"
    subprocess.run([_llvm_tool("llvm-objcopy"), "--dump-section=.hip_fatbin=" + fatbin, obj], check=True,
                   capture_output=True)
    subprocess.run([_llvm_tool("clang-offload-bundler"), "--unbundle", "--type=o", "--input=" + fatbin,
                    "--targets=hipv4-amdgcn-amd-amdhsa--" + ARCH, "--output=" + dev], check=True, capture_output=True)
    dis = subprocess.run([_llvm_tool("llvm-objdump"), "-d", dev], capture_output=True, text=True, check=True)
    count = 0
    for line in dis.stdout.splitlines():
        parts = line.split()
        if not parts or not parts[0].startswith(("v_", "s_", "ds_", "global_", "buffer_", "flat_")):
            continue
        count += 1
        if parts[0] in PACKED_FP32:
            raise RuntimeError("%s contains %s: packed-FP32 code generation was not disabled" % (obj, parts[0]))
    return count


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
        checked = list(ex.map(check_no_packed_fp32, objs))
    if verbose:
        print("device code checked: %d instructions, no packed-FP32 arithmetic" % sum(checked))
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
