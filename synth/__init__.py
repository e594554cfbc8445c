"""Seeded synthetic inputs (weights, KV caches, trees, tokens) shared by the
tests, the benchmark and the CPU reference.  Holds none of the decoding
method's arithmetic."""
from .configs import ModelShape, Workload, WORKLOADS, workload, T13B_SWEEP  # noqa: F401
