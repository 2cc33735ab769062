"""fp64 CPU oracle (test infrastructure only; never called by the HIP path)."""
