"""Seeded synthetic workloads (configs and input generators) for the
route-and-schedule tick. Shared by the oracle tests and the GPU path; it holds
no part of the tick's arithmetic."""
from . import configs, gen  # noqa: F401
