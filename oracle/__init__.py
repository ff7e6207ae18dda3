"""CPU oracle for the 3D-ResAttNet training step -- TEST INFRASTRUCTURE ONLY.

Plain, slow, float64 implementations of what the GPU path computes, written
from the definitions (see ``ops`` and ``net``).  Only the tests, the smoke
check and the CPU-baseline leg of the benchmark may import this package; the
product library never does, and the two share no code.  The only module both
sides use is the seeded input generator, which holds none of the method's
arithmetic.
"""
from . import ops, net  # noqa: F401
