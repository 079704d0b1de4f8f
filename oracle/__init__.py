"""Float64 CPU oracle for the DMC decode hot path (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library.
"""
from .dmc_oracle import (DMCOracle, LayerCache, UnitOracle, decision,  # noqa: F401
                         importance, sigmoid, OMEGA_FLOOR)
