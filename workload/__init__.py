"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle
checks.  Holds input generation only."""
from .configs import ORDER, WORKLOADS, Workload, describe  # noqa: F401
from .gen import Batch, heldout, make, manifest, window_seen  # noqa: F401
