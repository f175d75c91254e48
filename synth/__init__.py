"""Seeded synthetic workload generator shared by the oracle tests, the GPU tests and the bench.

Holds no part of the WnW method's arithmetic."""
from . import configs, gen  # noqa: F401
