"""Level-synchronous recursive inference on MI355X (gfx950).

Submodules:
  cortex   ctypes binding of libcortex.so (the C ABI of include/cortex.h)
  runner   device-side driver: upload a workload, enqueue linearize + forward
  inputs   seeded synthetic workloads (structure, inputs, weights)
  build    hipcc build of libcortex.so
"""
__all__ = ["cortex", "runner", "inputs", "build"]
