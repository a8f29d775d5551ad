"""Float64 CPU oracle for LUNA attention.  Test infrastructure only: imported by
the tests, the smoke check and the benchmark's CPU-baseline leg, never by the
GPU library."""
from .luna_oracle import *  # noqa: F401,F403
from . import luna_oracle  # noqa: F401
from . import luna_variants  # noqa: F401
from . import luna_distill  # noqa: F401
