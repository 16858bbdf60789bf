"""Seeded synthetic inputs for the PCED decode step (shared by the GPU path's tests,
the benchmark and the CPU oracle; holds no decoding arithmetic)."""
from . import counter, workloads  # noqa: F401
