"""Seeded synthetic workloads shared by the oracle and the GPU path (inputs only)."""
from . import rng, configs  # noqa: F401
