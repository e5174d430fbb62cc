"""Float64 CPU oracle of the GTF-DEER hot path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It shares no code with the HIP library.
"""
from .deer_oracle import *  # noqa: F401,F403
from . import brute  # noqa: F401
