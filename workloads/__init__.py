"""Seeded synthetic inputs shared by the oracle's tests and the GPU runs.

Holds the model tensor shapes, the five workload definitions and the counter-based
value generator (numpy here, HIP in ``csrc/fill.hip``).  Nothing in this package
computes any part of the allreduce.
"""
from . import configs, models, rng  # noqa: F401
