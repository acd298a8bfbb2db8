"""Seeded synthetic workloads shared by the tests, the smoke check and the bench.

This package holds none of the factorisation's arithmetic: it only draws
ratings (COO triplets) and initial factors.  Both the GPU path and the CPU
oracle receive its outputs as inputs.
"""
from .synth import CONFIGS, Workload, make, make_config, init_factors  # noqa: F401
