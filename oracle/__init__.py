"""CPU oracle (TEST INFRASTRUCTURE ONLY): the dense definition of the
Complementary Sparsity sparse-sparse layer, in float64/int64 numpy.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It shares no code with the GPU path.
"""
from . import cs_oracle, networks  # noqa: F401
