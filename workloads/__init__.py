"""Seeded synthetic workloads for the binary convolution (shapes + inputs)."""
from .configs import CONFIGS, CONFIG_NAMES, INT32_MAX, INT32_MIN, Layer, config
from .gen import LayerInputs, make_layer_inputs, random_words, rng_for, sha256

__all__ = [
    "CONFIGS", "CONFIG_NAMES", "INT32_MAX", "INT32_MIN", "Layer", "config",
    "LayerInputs", "make_layer_inputs", "random_words", "rng_for", "sha256",
]
