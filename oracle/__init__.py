"""CPU oracle for ShallowStream query-time evidence retrieval.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  The library path never calls it, and
it shares no code with the HIP implementation.

``oracle.oracle`` is the vectorised float64 reference (NumPy); ``oracle.brute``
is a second, independent pure-Python implementation for tiny inputs.
"""
from . import oracle, brute  # noqa: F401
