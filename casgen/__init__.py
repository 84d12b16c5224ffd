"""Seeded synthetic inputs for multi-cartridge prefix attention.

The one module whose outputs feed both the fp64 oracle and the GPU library:
shapes, seeded random bits and the benchmark configurations. No attention
arithmetic lives here.
"""
from . import rng  # noqa: F401
from .workloads import Workload, config, custom, make_tensors, packed, to_float  # noqa: F401
