"""CPU float64 oracle of the FNO spectral-convolution layer (test infrastructure).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package; the HIP library and its binding never do.
"""
from . import fno_oracle  # noqa: F401
