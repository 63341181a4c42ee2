"""CPU oracle for the K-VEC eviction step.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the CPU
baseline leg of the benchmark may import this package; the product library
never does, and the oracle never imports the product library.
"""
from .kvec_oracle import *  # noqa: F401,F403
