"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle."""
from .configs import WORKLOADS, Workload, make  # noqa: F401
