"""CPU oracle for Faster Flash Decoding decode attention (float64 numpy).

TEST INFRASTRUCTURE ONLY: imported by the tests, the package smoke check and the benchmark's
CPU-baseline leg, never by the product path.
"""
from .ffd_oracle import *  # noqa: F401,F403
