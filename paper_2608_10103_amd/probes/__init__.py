"""Hardware probes behind design choices of the kernels (not part of the GEMM path)."""
