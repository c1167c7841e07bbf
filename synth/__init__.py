"""Seeded synthetic workloads (configs + generator) shared by tests, bench and the oracle harness."""
from . import configs, generate  # noqa: F401
from .configs import CONFIGS, get  # noqa: F401
