"""Seeded synthetic inputs shared by the oracle and the GPU path.

This package holds workload descriptions (grid size, layer widths, batch,
schedule, hyper-parameters) and seeded dataset generators.  It contains none
of the coevolutionary method's arithmetic: both the oracle and the HIP path
consume what it produces, and neither imports the other.
"""
from .workloads import WORKLOADS, workload, small_workload  # noqa: F401
from .datasets import make_dataset  # noqa: F401
