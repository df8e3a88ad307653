"""CPU oracle for the Pr^2 MoE-layer hot path (test infrastructure).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its
Python binding) never imports, calls or loads it, and the two share no code.
See ``pr2_oracle`` for the definitions and the readings of the paper taken.
"""
from . import pr2_oracle  # noqa: F401
