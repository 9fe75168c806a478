"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle-side checks."""
from .configs import ALIASES, WORKLOADS, Workload, get  # noqa: F401
