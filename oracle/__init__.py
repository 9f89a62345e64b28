"""CPU oracle of the UltraMem memory-layer forward -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this package.
The GPU library never calls it and shares no code with it.
"""
from .umem_oracle import *  # noqa: F401,F403
