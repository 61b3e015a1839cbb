"""fp64 CPU oracle for the MLA-Online step.  TEST INFRASTRUCTURE ONLY: imported
by tests, the smoke check and the benchmark's CPU-baseline leg, never by the
library."""
from .mla_oracle import *  # noqa: F401,F403
from . import mla_oracle  # noqa: F401
