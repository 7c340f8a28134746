"""Seeded synthetic indexer workloads (queries, gates, keys) for the PIVOT indexer path.

This package only draws and encodes inputs; it holds none of the indexer's
arithmetic and is shared, unchanged, by the CPU oracle tests and by the HIP path.
"""
from .gen import WORKLOADS, Workload, make_prefill, make_decode, workload  # noqa: F401
