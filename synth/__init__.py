"""Seeded synthetic inputs for the CPDP path (host generator, device
generator binding, workloads).  Holds none of the method's arithmetic; shared
by the tests and the benchmark as the single source of input data."""
from . import gen, workloads  # noqa: F401
from .workloads import WORKLOADS, Workload  # noqa: F401
