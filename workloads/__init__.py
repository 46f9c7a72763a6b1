"""Seeded synthetic workloads (sizes, distributions and input generators).

Shared by the oracle, the tests and the benchmark; holds none of the
gradient-coding method's arithmetic.
"""
from .configs import ALL, BY_NAME, EXTRA, GRAPH, TINY, SMALL, HEADLINE, BANDWIDTH, LARGE, Workload  # noqa: F401
from . import gen  # noqa: F401
