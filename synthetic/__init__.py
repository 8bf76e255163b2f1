"""Seeded synthetic workloads (model shapes, random weights, KV prefill, start ids).

This module only draws random numbers and stores them as bf16; it holds none of the decode
step's arithmetic. Both the GPU library's tests/benchmark and the CPU oracle consume what it
produces, so neither side's inputs come from the other.
"""
from .configs import CONFIGS, get_config  # noqa: F401
from .inputs import make_weights, make_kv, make_start, Workload, make_workload, as_u16  # noqa: F401
