"""Plain CPU oracle for the MoE GEMM2 + combine stage and its partition
selector.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
baseline may import it; the product package never does, and the two share no
code (only the seeded input generator in ``workloads`` serves both).

Parity status: the combine result, the up-projection with its activation,
the selector arithmetic and the numeric helpers every comparison uses (bf16
widening, rel-L2, max-abs ratio) are pinned (tests/test_oracle_pins.py,
tests/test_layer_oracle.py, tests/test_selector_oracle.py,
tests/test_oracle_numeric_pins.py).  The absolute
time a candidate partition takes is not predicted in microseconds by the
paper, so wall-clock T(C) is "parity unpinned"; only the model's own
quantities are.
"""
from . import combine, layer, selector  # noqa: F401
