"""Helpers of the GPU parity tests: tensor transfer, error norms, and one-layer
graphs that run a chosen routine on the HIP path."""

import numpy as np

from oracle import numeric as O
from paper_2110_06037_amd import Graph, to_device
from workloads import to_f64

TOL = {"f32": 1e-4, "f16": 2e-2, "bf16": 2e-2}


def to_dev(arr, dtype):
    return to_device(arr, dtype, 0)


def from_dev(t, dtype):
    import torch
    t = t.detach().cpu()
    if dtype == "bf16":
        return to_f64(t.view(torch.int16).numpy().view(np.uint16), "bf16")
    return t.numpy().astype(np.float64)


def err(got, ref, dtype):
    """fp32: max abs error / max |ref|; f16/bf16: relative L2 over the tensor."""
    got = np.asarray(got, np.float64).reshape(-1)
    ref = np.asarray(ref, np.float64).reshape(-1)
    if dtype == "f32":
        return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


def single_layer_graph(dtype, in_shape, layer, w=None, b=None, layouts=None, algos=None,
                       params=True):
    n, c, h, wd = in_shape
    g = Graph(dtype, n, c, h, wd, device=0, layouts=layouts, algos=algos, params=params)
    g.add_spec(layer, w, b)
    return g


def run_routine(g, rid, x_dev, n_layers=2):
    ids = [0] * n_layers
    ids[-1] = rid
    g.set_path(ids)
    out = g.run(x_dev)
    import torch
    torch.cuda.synchronize()
    return out


def oracle_layer(layer, x, w, b, dtype):
    """Oracle output of one layer from stored inputs, rounded to the dtype."""
    xs = to_f64(x, dtype)
    ws = to_f64(w, dtype) if w is not None else None
    bs = b.astype(np.float64) if b is not None else None
    y = O.layer_forward(layer, [xs], ws, bs)
    return O.round_to(y, dtype)
