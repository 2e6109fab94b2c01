"""Seeded synthetic tensors for the workloads (shared input source of both sides).

Recipe: ``numpy.random.default_rng(seed)`` (PCG64).  Draw order: the input
tensor first, then for every layer in insertion order its weight, then its
bias (a further net input layer draws its tensor there instead).  Inputs are N(0, 1) or U[-1, 1] as the spec says; convolution and FC
weights are He-normal, std = sqrt(2 / fan_in) with fan_in = (C_in / groups)
* R * S (FC: in_features), untruncated; biases are U[-0.1, 0.1].  Values are
drawn in float64, then materialised in the run dtype by round-to-nearest-even
(biases in float32).  Both the oracle and the GPU path consume exactly these
bits; this module holds no arithmetic of the method itself.

bf16 tensors are carried as ``uint16`` bit patterns.
"""

from __future__ import annotations

import numpy as np

from .nets import channels

DTYPES = ("f32", "f16", "bf16")


def _round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64 -> bfloat16 bit patterns, one rounding, nearest-even.

    bfloat16 has 8 significant bits and the float32 exponent range
    (normal exponents -126..127, subnormal quantum 2**-133)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    flat = x.reshape(-1)
    o = out.reshape(-1)
    finite = np.isfinite(flat)
    v = flat.copy()
    v[~finite] = 0.0
    m, e = np.frexp(v)                     # v = m * 2**e, 0.5 <= |m| < 1
    # significant bits available at exponent e: 8 for normals, fewer for subnormals
    emin_norm = -125                       # frexp exponent of the smallest normal 2**-126
    prec_raw = np.where(e >= emin_norm, 8, 8 - (emin_norm - e))
    prec = np.maximum(prec_raw, 0)
    scaled = np.ldexp(m, prec)             # exact
    r = np.rint(scaled)                    # nearest-even
    r = np.where(prec_raw < 0, np.copysign(0.0, m), r)  # below half the smallest subnormal
    val = np.ldexp(r, e - prec)
    val = val.astype(np.float32)           # exact: val is representable in bf16 (or overflows)
    bits = val.view(np.uint32)
    hi = (bits >> 16).astype(np.uint16)
    over = np.abs(val.astype(np.float64)) > 3.3895313892515355e38
    hi = np.where(over, np.where(val < 0, np.uint16(0xFF80), np.uint16(0x7F80)), hi)
    hi = np.where(finite, hi, np.where(np.isnan(flat), np.uint16(0x7FC0),
                                       np.where(flat < 0, np.uint16(0xFF80), np.uint16(0x7F80))))
    o[:] = hi
    return out


def materialise(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage of ``dtype`` (RNE)."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "f16":
        return x.astype(np.float16)        # numpy converts float64 -> half in one rounding
    if dtype == "bf16":
        return _round_bf16_bits(x)
    raise ValueError(dtype)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored values of ``dtype`` to float64 (exact)."""
    if dtype == "bf16":
        a = np.asarray(a, dtype=np.uint16)
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a).astype(np.float64)


def weight_shapes(spec):
    """(weight shape, bias length) per layer; None for layers without weights."""
    ch = channels(spec)
    out = []
    for layer in spec["layers"]:
        t = layer["type"]
        if t == "input":
            out.append(None)
            continue
        cin = ch[layer["in"][0]]
        if t == "conv":
            g = layer["groups"]
            if layer.get("proj"):  # and the projected shortcut's 1x1 weights
                out.append(((layer["k"], cin // g, layer["r"], layer["s"]), layer["k"],
                            (layer["k"], ch[layer["in"][1]], 1, 1)))
            else:
                out.append(((layer["k"], cin // g, layer["r"], layer["s"]), layer["k"]))
        elif t == "fc":
            out.append(((layer["k"], cin), layer["k"]))
        else:
            out.append(None)
    return out


def generate(spec, seed=None):
    """Draw the input, weights and biases of ``spec``.

    Returns a dict with ``x`` (N x C x H x W, stored dtype), ``w`` and ``b``
    (lists indexed by layer id - 1; None for layers without weights; weights in
    the stored dtype, biases float32) and ``inputs`` ({layer id: tensor} of the
    further net inputs)."""
    dtype = spec["dtype"]
    rng = np.random.default_rng(spec.get("seed", 0) if seed is None else seed)
    n = spec["batch"]
    c, h, w = spec["in_chw"]

    def draw_input(shape):
        if spec["input_dist"] == "normal":
            return rng.standard_normal(shape)
        return rng.uniform(-1.0, 1.0, shape)

    x = draw_input((n, c, h, w))
    ws, bs = [], []
    extra = {}
    for i, (layer, shp) in enumerate(zip(spec["layers"], weight_shapes(spec)), start=1):
        if layer["type"] == "input":
            extra[i] = materialise(draw_input((n, *layer["chw"])), dtype)
            ws.append(None)
            bs.append(None)
            continue
        if shp is None:
            ws.append(None)
            bs.append(None)
            continue
        wshape, k = shp[:2]
        fan_in = int(np.prod(wshape[1:]))
        wt = rng.standard_normal(wshape) * np.sqrt(2.0 / fan_in)
        bt = rng.uniform(-0.1, 0.1, k)
        if len(shp) == 3:  # a projected shortcut: its weights and bias follow
            pshape = shp[2]
            wp = rng.standard_normal(pshape) * np.sqrt(2.0 / int(np.prod(pshape[1:])))
            bp = rng.uniform(-0.1, 0.1, k)
            ws.append((materialise(wt, dtype), materialise(wp, dtype)))
            bs.append((bt.astype(np.float32), bp.astype(np.float32)))
            continue
        ws.append(materialise(wt, dtype))
        bs.append(bt.astype(np.float32))
    return {"x": materialise(x, dtype), "w": ws, "b": bs, "inputs": extra, "dtype": dtype}


def random_tensor(shape, dtype, seed, dist="uniform", scale=1.0):
    """A single seeded tensor, for per-routine tests."""
    rng = np.random.default_rng(seed)
    if dist == "normal":
        v = rng.standard_normal(shape) * scale
    elif dist == "int":
        v = rng.integers(-1, 2, size=shape).astype(np.float64) * scale
    else:
        v = rng.uniform(-scale, scale, shape)
    return materialise(v, dtype)


def decode(tensors, dtype):
    """The generated tensors in float64: the input, the weights (pairs for a
    projected shortcut's layer stay pairs), the biases and further inputs."""
    def dec(v, f):
        if v is None:
            return None
        return tuple(f(e) for e in v) if isinstance(v, tuple) else f(v)
    return {"x": to_f64(tensors["x"], dtype),
            "w": [dec(w, lambda e: to_f64(e, dtype)) for w in tensors["w"]],
            "b": [dec(b, lambda e: e.astype(np.float64)) for b in tensors["b"]],
            "inputs": {k: to_f64(v, dtype) for k, v in tensors.get("inputs", {}).items()}}
