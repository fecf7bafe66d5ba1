"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

This package draws the synthetic prefill K/V caches, probe queries, decode
queries and fixed head-mode assignments that stand in for a real model's
cache.  It contains none of the compression method's arithmetic (no depth
transform, no top-k, no routing loss, no attention): only random draws, the
inter-layer correlation recipe of the workloads, planted needle spikes and
rounding of the drawn values to the storage precision.
"""
from .workloads import WORKLOADS, Workload, scaled  # noqa: F401
from . import gen  # noqa: F401
