"""Seeded synthetic inputs for the TASP decode path (weights, caches, activations, masks).

This package is the only code that the CPU oracle, the GPU parity tests and the benchmark
share. It draws random numbers, quantises the drawn weights into the INT8 store format, rounds
drawn values to BF16, and draws masks. It contains none of the decode path's arithmetic.
"""
from .gen import *  # noqa: F401,F403
from .configs import *  # noqa: F401,F403
