"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds shapes, seeds, random draws and bf16 bit packing only. It
contains none of the layer's arithmetic: both the fp64 oracle and the HIP path
consume what it produces, and neither depends on the other through it.
"""
from .configs import CONFIGS, LayerShape, Workload, get  # noqa: F401
from . import gen  # noqa: F401
