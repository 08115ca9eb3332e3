"""CPU oracle for TP-aware dequantization: test infrastructure only.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package. The product path (the HIP library and its binding) never does.
"""
from .tpdq_oracle import *  # noqa: F401,F403
from . import tpdq_oracle  # noqa: F401
