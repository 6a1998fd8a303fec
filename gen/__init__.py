"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This package holds no PAR, routing or attention arithmetic: it only draws
random tensors with the shapes, value distributions and structure of the
paper's two backbones (Matrix-Game-like and HY-World-like blocks) and of two
stress cases.  Both the HIP path and the oracle consume its outputs.
"""
from .workloads import (  # noqa: F401
    Workload, WORKLOADS, get, attn_inputs, par_inputs, seeds_for, wo_weight, control_inputs,
)
