"""MI355X-native routine-selection CNN inference (SoftNeuro's method).

Layers have several interchangeable routines (direct, implicit-GEMM and
Winograd convolution in NCHW, NHWC or NC8HW8 layouts, plus layout converters);
every routine is profiled on the GPU and a dynamic program over the layer
graph (DPRS) selects the fastest routine path including conversion costs.
The work is done by libsoftneuro.so (C ABI in include/softneuro.h, HIP
kernels for gfx950); this package is its Python binding.
"""

from .graph import Graph, build_from_spec, to_device
from . import native

__all__ = ["Graph", "build_from_spec", "to_device", "native"]
