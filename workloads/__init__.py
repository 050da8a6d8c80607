"""Seeded synthetic inputs for the bounded-state restore path.

This package describes and generates the workloads only: token IDs, the
per-(chunk, group) KV payload bytes held by the external tier, destination
block tables, pool sentinels, initial valid bytes and failure-injection
points.  It contains none of the restore method's arithmetic (no hashing, no
slot layout, no block mapping, no tags); both the CPU oracle and the HIP path
consume what it produces.
"""

from .configs import CONFIGS, GroupSpec, Workload, get_config  # noqa: F401
from .gen import WorkloadInputs, generate  # noqa: F401
