"""Plain float64 CPU oracle for the GRKV value-step compression path.

Test infrastructure only: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .grkv_oracle import *  # noqa: F401,F403
from .grkv_oracle import __all__  # noqa: F401
