"""Seeded synthetic workloads for the streaming beam-search decoder.

This package only draws random numbers and lays them out; it holds none of the
search arithmetic. Both the fp64 oracle and the HIP path read their inputs from
here, so the two sides see bit-identical weights and per-input data.
"""
from .configs import CONFIGS, SearchConfig, get_config, scaled
from .gen import Workload, make_workload, bf16_bits_to_f32

__all__ = ["CONFIGS", "SearchConfig", "get_config", "scaled", "Workload",
           "make_workload", "bf16_bits_to_f32"]
