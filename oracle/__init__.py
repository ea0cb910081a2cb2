"""fp64 CPU oracle for the FPO hot path (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product path (the HIP library and its binding) never
calls it, and it shares no code with that path.
"""
from .fpo_oracle import *  # noqa: F401,F403
