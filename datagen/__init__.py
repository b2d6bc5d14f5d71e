"""Seeded synthetic inputs shaped like DReSD's datastores.

This package is shared by the tests, the smoke check and the benchmark.  It
holds no retrieval arithmetic: it only draws keys, continuations and queries
with fixed seeds, so the oracle and the device path read the same bytes.
"""
from .workloads import WORKLOADS, Workload, generate, to_numpy_bits  # noqa: F401
