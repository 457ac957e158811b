"""fp64 CPU oracle for the Video Delta Attention forward pass.

TEST INFRASTRUCTURE ONLY: imported by the test-suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .vda_oracle import *  # noqa: F401,F403
from .vda_oracle import RMS_EPS  # noqa: F401
