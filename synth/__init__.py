"""Seeded synthetic inputs shared by the tests, the bench and the oracle checks.

This package draws random inputs and plants known structure in them; it holds
none of the method's arithmetic (no attention, no expansion, no acceptance).
"""

from .workloads import WORKLOADS, Workload  # noqa: F401
