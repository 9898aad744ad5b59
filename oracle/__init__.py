"""fp64 CPU oracle of (n,k) MDS-coded matrix multiplication (test infrastructure).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library: the only module
both sides use is `synth`, the seeded input generator.
"""
from . import coded  # noqa: F401
