"""Seeded synthetic sparse 1x1-convolution layers.

This package only draws inputs: sparsity masks, weight values, biases and
activations.  It holds none of the method's arithmetic, so both the CPU
oracle (``oracle/``) and the GPU library (``paper_1911_09723_amd``) can be
fed from it without sharing any computation.
"""

from .layers import Layer, make_layer, make_depthwise, densify, expand_blocks_to_csr
from .configs import CONFIGS, config_layers, layer_seed, TARGET
from .mobilenet import MBV1_BLOCKS, MobileNetV1, make_mobilenet_v1, make_image

__all__ = [
    "Layer",
    "make_layer",
    "make_depthwise",
    "densify",
    "expand_blocks_to_csr",
    "CONFIGS",
    "config_layers",
    "layer_seed",
    "TARGET",
    "MBV1_BLOCKS",
    "MobileNetV1",
    "make_mobilenet_v1",
    "make_image",
]
