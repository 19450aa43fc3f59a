"""Seeded synthetic workloads shaped like the paper's agent contexts.

Input generation only: shapes, lengths, values and page placements.  No
attention or paging arithmetic lives here, so the oracle and the device path
can both consume these inputs.
"""
from .configs import Workload, AssembleInputs, make, CONFIGS  # noqa: F401
from . import rng  # noqa: F401
