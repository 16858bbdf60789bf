"""CPU oracle for the PCED decode step.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the package's smoke check and
by the benchmark's CPU-baseline leg; never by the product path. It shares no code
with the GPU path.
"""
