"""Seeded synthetic inputs for the kNN-LM mixture step.

This package only draws random inputs (keys, queries, value tokens, p_LM rows,
key-set offsets).  It holds none of the method's arithmetic, and both the HIP
path and the CPU oracle consume what it produces.
"""
from .gen import (  # noqa: F401
    Spec,
    Workload,
    CONFIGS,
    config,
    make,
    zipf_cdf,
)
