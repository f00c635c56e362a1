"""Seeded synthetic workloads and input generators (no arithmetic of the method)."""
from .configs import PAGE, Workload, workload  # noqa: F401
from . import gen  # noqa: F401
