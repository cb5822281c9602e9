"""Seeded synthetic workloads (shapes, batch recipes, input generators).

Shared by the oracle's tests, the device tests and the benchmark.  It holds
none of the decode step's arithmetic.
"""
from . import gen, configs  # noqa: F401
