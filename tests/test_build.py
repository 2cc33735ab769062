"""The build's device-code check (no GPU needed): a gfx950 object compiled
without the packed-FP32 switch is rejected, the same source compiled with the
build's flags passes."""
import os
import shutil

import pytest

from paper_2011_01383_amd import build as B

SRC = r'''
#include <hip/hip_runtime.h>
__global__ void axpy2(float2 *a, const float2 *b, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    float2 x = a[i], y = b[i];
    x.x = x.x * y.x + 1.0f;
    x.y = x.y * y.y + 1.0f;
    a[i] = x;
  }
}
'''


def _compile(tmp_path, flags, name):
    import subprocess
    src = tmp_path / "pk.hip"
    src.write_text(SRC)
    obj = str(tmp_path / name)
    subprocess.run([B._hipcc(), "-O3", "--offload-arch=" + B.ARCH, *flags, "-c", str(src), "-o", obj],
                   check=True, capture_output=True)
    return obj


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not installed")
def test_packed_fp32_check(tmp_path):
    plain = _compile(tmp_path, [], "plain.o")
    with pytest.raises(RuntimeError, match="packed-FP32"):
        B.check_no_packed_fp32(plain)
    flagged = _compile(tmp_path, [f for f in B.HIPCC_FLAGS if not f.startswith("--offload-arch")], "flagged.o")
    assert B.check_no_packed_fp32(flagged) > 0
