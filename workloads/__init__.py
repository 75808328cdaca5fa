"""Seeded synthetic decode workloads (inputs only; no Top-K arithmetic here).

Both the GPU path's tests/benchmark and the oracle consume these buffers; the
module holds none of the method's arithmetic.
"""
from .decode import CONFIGS, Workload, generate, spec  # noqa: F401
