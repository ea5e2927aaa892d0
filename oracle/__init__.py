"""CPU oracle of SpecPrefetch's offloaded-MoE decode hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 numpy
restatement of what the method computes, used to check the device path.  Only
the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path (the HIP library and its Python binding) never
does, and shares no code with it.  The only module both sides read is
``workload`` (seeded inputs, no arithmetic of the method).

Parity pins: every function is checked in ``tests/test_oracle_pins.py``
against something other than itself (brute force, closed forms, independent
library routines, invariants, a hand-worked cache trace).
"""
from .spp_oracle import *  # noqa: F401,F403
