"""Seeded synthetic inputs shared by the oracle-side tests and the HIP path (inputs only)."""

from . import trees, configs  # noqa: F401
from .configs import WORKLOADS, Workload, round_inputs  # noqa: F401
