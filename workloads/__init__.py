"""Seeded synthetic inputs for the WUSH-KV hot path (tests and benchmark).

Holds none of the method's arithmetic: it only draws keys, values, queries
and transforms with the shapes and distributions of the paper's workloads.
"""
from .synth import CONFIGS, Workload, make_rng, make_transform, random_orthogonal, rope  # noqa: F401
