"""CPU oracle for the MicroMix hot path.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .mx_oracle import *  # noqa: F401,F403
