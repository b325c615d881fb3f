"""CPU oracle for paged graph beam search -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library shares no code with it.
"""
from .oracle import Oracle, build, load, LIB_PATH, SRC_PATH

__all__ = ["Oracle", "build", "load", "LIB_PATH", "SRC_PATH"]
