"""Seeded synthetic workloads shared by the HIP path's tests/benchmark and the CPU oracle.

This package only draws numbers: it holds none of the method's arithmetic (no
projection, selection, attention or MLP code), so that both sides can consume the
same stored values without sharing any computation.
"""
from .configs import CONFIGS, Config, get_config
from .gen import make_layer, zipf_mlp_sets, uniform_head_sets, to_numpy64

__all__ = ["CONFIGS", "Config", "get_config", "make_layer", "zipf_mlp_sets",
           "uniform_head_sets", "to_numpy64"]
