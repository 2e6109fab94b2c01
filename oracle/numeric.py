"""Numerical oracle: float64 forward pass of a net, layer by layer.

TEST INFRASTRUCTURE ONLY (tests, the smoke check and the benchmark's CPU
baseline).  The arithmetic lives in ``sn_oracle.c``; this module marshals
arrays and infers shapes.  Each layer computes the plain definition of its
type (paper Sec. III-B: a net is a DAG of layers exchanging blobs; the
routines chosen for a layer do not change what it computes).

Storage modes: ``"dtype"`` rounds every layer output once from float64 to the
run dtype (nearest-even), which is what any GPU routine must store;
``"f64"`` keeps exact values.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build_oracle

_DT = {"f32": 0, "f16": 1, "bf16": 2}
_ACT = {"none": 0, "relu": 1, "relu6": 2}
_lib = None


def lib():
    global _lib
    if _lib is None:
        path = build_oracle.build(force=False)
        L = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        i = ctypes.c_int
        L.or_conv2d.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, i, dp, i, dp]
        L.or_conv2d_points.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, i, dp, i,
                                       ctypes.POINTER(ctypes.c_int64), ctypes.c_int64, dp]
        L.or_maxpool.argtypes = [dp, i, i, i, i, i, i, i, dp]
        L.or_gap.argtypes = [dp, i, i, i, i, dp]
        L.or_add.argtypes = [dp, dp, ctypes.c_int64, i, dp]
        L.or_fc.argtypes = [dp, i, i, dp, i, dp, dp]
        L.or_round.argtypes = [dp, ctypes.c_int64, i]
        L.or_round1.argtypes = [ctypes.c_double, i]
        L.or_round1.restype = ctypes.c_double
        L.or_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def out_hw(h, w, r, s, stride, pad):
    return (h + 2 * pad - r) // stride + 1, (w + 2 * pad - s) // stride + 1


def conv2d(x, w, b, stride=1, pad=0, groups=1, act="none"):
    x, w = _f64(x), _f64(w)
    n, c, h, wd = x.shape
    k, cg, r, s = w.shape
    assert cg * groups == c and k % groups == 0
    p, q = out_hw(h, wd, r, s, stride, pad)
    y = np.empty((n, k, p, q))
    bb = _f64(b) if b is not None else None
    lib().or_conv2d(_p(x), n, c, h, wd, _p(w), k, r, s, stride, pad, groups,
                    _p(bb) if bb is not None else None, _ACT[act], _p(y))
    return y


def conv2d_points(x, w, b, idx, stride=1, pad=0, groups=1, act="none"):
    """Oracle values at sampled output positions idx[i] = (n, k, p, q)."""
    x, w = _f64(x), _f64(w)
    n, c, h, wd = x.shape
    k, cg, r, s = w.shape
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(len(idx))
    bb = _f64(b) if b is not None else None
    lib().or_conv2d_points(_p(x), n, c, h, wd, _p(w), k, r, s, stride, pad, groups,
                           _p(bb) if bb is not None else None, _ACT[act],
                           idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), len(idx), _p(out))
    return out


def maxpool(x, k=3, stride=2, pad=1):
    x = _f64(x)
    n, c, h, w = x.shape
    p, q = out_hw(h, w, k, k, stride, pad)
    y = np.empty((n, c, p, q))
    lib().or_maxpool(_p(x), n, c, h, w, k, stride, pad, _p(y))
    return y


def gap(x):
    x = _f64(x)
    n, c, h, w = x.shape
    y = np.empty((n, c, 1, 1))
    lib().or_gap(_p(x), n, c, h, w, _p(y))
    return y


def add(a, b, act="none"):
    a, b = _f64(a), _f64(b)
    assert a.shape == b.shape
    y = np.empty_like(a)
    lib().or_add(_p(a), _p(b), a.size, _ACT[act], _p(y))
    return y


def activate(y, act):
    """The fused activations: identity, ReLU = max(y, 0), ReLU6 = min(max(y, 0), 6)."""
    y = _f64(y)
    if act == "relu":
        return np.maximum(y, 0.0)
    if act == "relu6":
        return np.minimum(np.maximum(y, 0.0), 6.0)
    assert act == "none", act
    return y.copy()


def fc(x, w, b):
    x, w = _f64(x), _f64(w)
    n = x.shape[0]
    xin = x.reshape(n, -1)
    k, cin = w.shape
    assert xin.shape[1] == cin
    y = np.empty((n, k))
    bb = _f64(b) if b is not None else None
    lib().or_fc(_p(np.ascontiguousarray(xin)), n, cin, _p(w), k,
                _p(bb) if bb is not None else None, _p(y))
    return y.reshape(n, k, 1, 1)


def round_to(a, dtype):
    """Storage rounding of float64 values to ``dtype`` (one rounding, nearest-even)."""
    a = np.array(a, dtype=np.float64, copy=True)
    lib().or_round(_p(a), a.size, _DT[dtype])
    return a


def layer_forward(layer, inputs, w=None, b=None):
    t = layer["type"]
    if t == "conv":
        if layer.get("proj"):
            # projected shortcut (a bottleneck block's residual add with its
            # 1x1 projection, folded into the convolution): the two
            # convolutions and their biases summed, then the activation
            (wm, wp), (bm, bp) = w, b
            y = conv2d(inputs[0], wm, bm, layer["stride"], layer["pad"], 1, "none")
            y = y + conv2d(inputs[1], wp, bp, layer["proj"]["stride"], 0, 1, "none")
            return activate(y, layer["act"])
        if len(inputs) > 1:  # residual added before the activation
            y = conv2d(inputs[0], w, b, layer["stride"], layer["pad"], layer["groups"], "none")
            return add(y, inputs[1], layer["act"])
        return conv2d(inputs[0], w, b, layer["stride"], layer["pad"], layer["groups"],
                      layer["act"])
    if t == "maxpool":
        return maxpool(inputs[0], layer["k"], layer["stride"], layer["pad"])
    if t == "gap":
        return gap(inputs[0])
    if t == "add":
        return add(inputs[0], inputs[1], layer.get("act", "none"))
    if t == "fc":
        return activate(fc(inputs[0], w, b), layer.get("act", "none"))
    raise ValueError(t)


def forward(spec, tensors, storage="dtype", keep=None, layer_dtypes=None):
    """Run the whole net.  ``tensors`` comes from ``workloads.generate`` decoded to
    float64 (keys x, w, b, and ``inputs`` {layer id: tensor} for further net
    inputs).  Returns the list of layer outputs (index 0 = input);
    intermediate outputs no longer needed are dropped unless ``keep`` is True
    (net outputs listed in ``spec["outputs"]`` are always kept).

    ``layer_dtypes`` (storage "dtype" only): the element type each layer
    computes in, a list indexed by layer id (entries for input layers are
    ignored; default: the spec's dtype everywhere).  This is the oracle of a
    precision-hybrid path (Sec. IV-F): a layer reads every input cast to its
    own type (the adapt between schemas, one rounding of the stored value),
    uses the caller's weights rounded once to its type (biases stay float32),
    and stores its output rounded to its type; the net outputs are cast back
    to the spec's dtype."""
    dtype = spec["dtype"]
    layers = spec["layers"]
    ldt = [dtype] * (len(layers) + 1)
    if layer_dtypes is not None:
        assert storage == "dtype" and len(layer_dtypes) == len(layers) + 1
        for i, L in enumerate(layers, start=1):
            if L["type"] != "input":
                ldt[i] = layer_dtypes[i]
    keep_ids = set(spec.get("outputs", [len(layers)]))
    last_use = {}
    for i, layer in enumerate(layers, start=1):
        for j in layer["in"]:
            last_use[j] = i
    outs = [None] * (len(layers) + 1)
    outs[0] = _f64(tensors["x"])
    for i, layer in enumerate(layers, start=1):
        if layer["type"] == "input":
            outs[i] = _f64(tensors["inputs"][i])
            continue
        ins = [outs[j] for j in layer["in"]]
        w = tensors["w"][i - 1]
        if storage == "dtype":
            ins = [x if ldt[j] == ldt[i] else round_to(x, ldt[i]) for x, j in zip(ins, layer["in"])]
            if ldt[i] != dtype and w is not None:
                w = tuple(round_to(v, ldt[i]) for v in w) if isinstance(w, tuple) else round_to(w, ldt[i])
        y = layer_forward(layer, ins, w, tensors["b"][i - 1])
        if storage == "dtype":
            y = round_to(y, ldt[i])
        outs[i] = y
        if not keep:
            for j in layer["in"]:
                if last_use.get(j) == i and j != 0 and j not in keep_ids:
                    outs[j] = None
    if storage == "dtype":
        for o in keep_ids:
            if ldt[o] != dtype:
                outs[o] = round_to(outs[o], dtype)
    return outs


def num_threads():
    return lib().or_num_threads()
