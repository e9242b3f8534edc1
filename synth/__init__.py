"""Seeded synthetic inputs for one UniF-MoE feed-forward layer.

This module is shared by the CPU oracle, the tests and the benchmark. It only
draws random numbers and lays them out; it holds none of the layer's
arithmetic (no routing, no expert evaluation). Constants that depend on the
layer's routing (router scales for two workloads) are read from
``calibration.json``, which ``oracle/calibrate.py`` writes.
"""
from .configs import CONFIGS, config_names, get_config, layer_config
from .generate import generate, block_inputs, upstream_grad, bf16_bits_to_f32, f32_to_bf16_bits

__all__ = [
    "CONFIGS", "config_names", "get_config", "layer_config", "generate", "block_inputs", "upstream_grad",
    "bf16_bits_to_f32", "f32_to_bf16_bits",
]
