"""Seeded synthetic inputs for the VSD path-scoring workloads.

The paper trains on ShareGPT / OpenThoughts / LLaVA-Instruct positions with
EAGLE-3 / MSD draft heads over Vicuna (32 000-token) and LLaMA-3 (128 256-token)
vocabularies.  Those datasets and weights are not used: these generators make
logits of the same shapes and of controlled distribution instead.  This module
holds none of the method's arithmetic; it only draws inputs, and both the
library's tests and the oracle's consume what it returns.
"""
from .configs import CONFIGS, Config, get_config, scaled
from .gen import make_inputs, make_inputs_numpy_c1, positions_rows
from .rollout import context_rows, depth_view, make_tables

__all__ = ["CONFIGS", "Config", "get_config", "scaled", "make_inputs",
           "make_inputs_numpy_c1", "positions_rows", "context_rows", "depth_view", "make_tables"]
