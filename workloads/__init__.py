"""Workload shapes (segment tables) and seeded synthetic inputs.

Shared by the tests, the benchmark and the smoke check; imports neither the
oracle nor the HIP package and holds none of the method's arithmetic."""
from . import gen, tables  # noqa: F401
