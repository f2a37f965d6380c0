"""CPU oracle for the NVFP4 hot path.  TEST INFRASTRUCTURE ONLY: imported by
tests/, the smoke check and the benchmark's CPU-baseline leg, never by the
library."""
from .nvfp4 import *  # noqa: F401,F403
