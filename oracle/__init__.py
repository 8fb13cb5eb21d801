"""CPU oracle for the in-memory snapshot path (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  The product library never does.
"""
from .oracle import *  # noqa: F401,F403
