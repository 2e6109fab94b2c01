"""Synthetic workloads: network structures and seeded tensors.

This package is the one input source shared by the oracle and the GPU path;
it contains no arithmetic of the method (no convolution, no path selection).
"""

from .nets import (all_configs, channels, conv_sweep, edges, fuse_projection, fuse_residual, mobilenet_v2, net_d, resnet18,
                   resnet50, tiny_chain, vgg16, with_batch, CONV_SWEEP_SHAPES)
from .gen import decode, generate, materialise, random_tensor, to_f64, weight_shapes

__all__ = ["all_configs", "channels", "conv_sweep", "decode", "edges", "fuse_projection", "fuse_residual",
           "mobilenet_v2", "net_d", "resnet18", "resnet50", "tiny_chain", "vgg16", "with_batch",
           "CONV_SWEEP_SHAPES", "generate", "materialise", "random_tensor", "to_f64", "weight_shapes"]
