"""Float64 CPU oracle for MRA-2 attention.

Test infrastructure: only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it. The product path never does.
"""
from . import mra_oracle  # noqa: F401
