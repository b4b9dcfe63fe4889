"""CPU oracle for the RRS W4A4 linear layer (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use it.
"""
from . import rrs_oracle  # noqa: F401
