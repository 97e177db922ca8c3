"""Seeded synthetic workloads shared by the HIP path's tests/benchmark and the CPU oracle.

This package only draws numbers and stores them (including as 4-bit blocks, the
W4A16 input format): it holds none of the method's arithmetic (no dequantisation,
projection, selection, attention or MLP code), so that both sides can consume the
same stored values without sharing any computation.
"""
from .configs import CONFIGS, Config, get_config
from .gen import make_layer, quantize_q4, zipf_mlp_sets, uniform_head_sets, to_numpy64

__all__ = ["CONFIGS", "Config", "get_config", "make_layer", "quantize_q4", "zipf_mlp_sets",
           "uniform_head_sets", "to_numpy64"]
