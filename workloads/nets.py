"""Network specifications of the synthetic workloads (structure only, no arithmetic).

A net is a DAG of layers in insertion (= topological) order.  Layer 0 is the
auxiliary input layer that carries the user's N x C x H x W tensor (the
paper's auxiliary input layer, Sec. IV-E); layers 1..n are listed in
``spec["layers"]`` and the last one is the net output.  Each layer is a dict:

* ``{"type": "conv", "in": [j], "k": K, "r": R, "s": S, "stride": st,
  "pad": p, "groups": g, "act": "none"|"relu"|"relu6"}`` -- 2-D convolution
  (cross-correlation) with a fused activation; ``groups`` is 1 (dense) or the
  channel count (depthwise).  ``"in": [j, r]`` adds layer r's output (a
  residual of the output's shape) before the activation.  Batch-norm layers of the original models are
  taken as folded into the convolution bias, as the paper's importer does
  when it fuses BN and ReLU into the preceding layer (Sec. III-A).
* ``{"type": "maxpool", "in": [j], "k": 3, "stride": 2, "pad": 1}``
* ``{"type": "gap", "in": [j]}`` -- global average pooling to N x C x 1 x 1.
* ``{"type": "add", "in": [a, b], "act": ...}`` -- residual merge.
* ``{"type": "fc", "in": [j], "k": out, "act": ...}`` -- dense layer,
  y = act(W x + b) on an N x C x 1 x 1 input ("act" optional, default none).
* ``{"type": "input", "in": [], "chw": [C, H, W]}`` -- a further net input
  (batch N of the spec); ``spec["outputs"]`` (optional) lists the net
  outputs in order, else the last layer is the one output (Sec. IV-E).

The shapes follow the model families the paper evaluates (Sec. V: ResNet50,
MobileNetV2, VGG16; ResNet-18 and a tiny chain are smaller members of the
same families).  Weights are random (He-normal) since no trained model is used.
"""

from __future__ import annotations

import copy

ACTS = ("none", "relu", "relu6")


def _conv(inp, k, r, stride=1, pad=None, groups=1, act="none"):
    if pad is None:
        pad = r // 2
    return {"type": "conv", "in": [inp], "k": k, "r": r, "s": r, "stride": stride,
            "pad": pad, "groups": groups, "act": act}


class _Builder:
    def __init__(self):
        self.layers = []

    def add(self, layer):
        self.layers.append(layer)
        return len(self.layers)          # id of the new layer (input is 0)


def tiny_chain():
    """Tiny fp32 chain: conv3x3 3->16 +ReLU, conv3x3 16->32 /2 +ReLU,
    conv1x1 32->32, global average pool, FC 32->10 on a 1x3x32x32 input."""
    b = _Builder()
    x = b.add(_conv(0, 16, 3, 1, 1, act="relu"))
    x = b.add(_conv(x, 32, 3, 2, 1, act="relu"))
    x = b.add(_conv(x, 32, 1, 1, 0))
    x = b.add({"type": "gap", "in": [x]})
    b.add({"type": "fc", "in": [x], "k": 10})
    return {"name": "tiny_chain", "dtype": "f32", "batch": 1, "in_chw": [3, 32, 32],
            "input_dist": "normal", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC"], "algos": ["direct", "igemm"]}


def conv_sweep(c, hw, batch=32, dtype="f16"):
    """One 3x3 stride-1 pad-1 convolution C->C at H=W=hw (the cost-table sweep)."""
    b = _Builder()
    b.add(_conv(0, c, 3, 1, 1))
    return {"name": f"conv3x3_c{c}_hw{hw}", "dtype": dtype, "batch": batch,
            "in_chw": [c, hw, hw], "input_dist": "uniform", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


CONV_SWEEP_SHAPES = [(64, 56), (128, 28), (256, 14), (512, 7)]


def _stem_resnet(b):
    x = b.add(_conv(0, 64, 7, 2, 3, act="relu"))
    return b.add({"type": "maxpool", "in": [x], "k": 3, "stride": 2, "pad": 1})


def resnet18(batch=1, dtype="bf16"):
    """ResNet-18 shape: basic blocks [2,2,2,2], widths 64..512, 1x1/2 projections."""
    b = _Builder()
    x = _stem_resnet(b)
    cin = 64
    for stage, width in enumerate([64, 128, 256, 512]):
        for blk in range(2):
            stride = 2 if (stage > 0 and blk == 0) else 1
            inp = x
            y = b.add(_conv(inp, width, 3, stride, 1, act="relu"))
            y = b.add(_conv(y, width, 3, 1, 1))
            sc = inp
            if stride != 1 or cin != width:
                sc = b.add(_conv(inp, width, 1, stride, 0))
            x = b.add({"type": "add", "in": [y, sc], "act": "relu"})
            cin = width
    x = b.add({"type": "gap", "in": [x]})
    b.add({"type": "fc", "in": [x], "k": 1000})
    return {"name": f"resnet18_bs{batch}", "dtype": dtype, "batch": batch,
            "in_chw": [3, 224, 224], "input_dist": "uniform", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


def resnet50(batch=1, dtype="bf16"):
    """ResNet-50 shape (v1.5: stride on the 3x3): bottlenecks [3,4,6,3], mid
    widths 64..512 with x4 expansion, projection shortcuts, FC 2048->1000."""
    b = _Builder()
    x = _stem_resnet(b)
    cin = 64
    for stage, (mid, nblk) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        for blk in range(nblk):
            stride = 2 if (stage > 0 and blk == 0) else 1
            inp = x
            y = b.add(_conv(inp, mid, 1, 1, 0, act="relu"))
            y = b.add(_conv(y, mid, 3, stride, 1, act="relu"))
            y = b.add(_conv(y, 4 * mid, 1, 1, 0))
            sc = inp
            if blk == 0:
                sc = b.add(_conv(inp, 4 * mid, 1, stride, 0))
            x = b.add({"type": "add", "in": [y, sc], "act": "relu"})
            cin = 4 * mid
    x = b.add({"type": "gap", "in": [x]})
    b.add({"type": "fc", "in": [x], "k": 1000})
    return {"name": f"resnet50_bs{batch}_{dtype}", "dtype": dtype, "batch": batch,
            "in_chw": [3, 224, 224], "input_dist": "uniform", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


MBV2_SCHEDULE = [  # (expansion t, out channels c, repeats n, first stride s)
    (1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
    (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1)]


def mobilenet_v2(batch=1, dtype="bf16", first_t=1):
    """MobileNetV2 shape: 3x3/2 stem 32, 17 inverted-residual blocks (1x1
    expand + ReLU6, depthwise 3x3 + ReLU6, linear 1x1 project, residual when
    stride 1 and C_in == C_out), 1x1 conv 1280, average pool, FC 1280->1000."""
    b = _Builder()
    x = b.add(_conv(0, 32, 3, 2, 1, act="relu6"))
    cin = 32
    for i, (t, c, n, s) in enumerate(MBV2_SCHEDULE):
        if i == 0:
            t = first_t
        for blk in range(n):
            stride = s if blk == 0 else 1
            inp = x
            hid = cin * t
            y = inp
            if t != 1:
                y = b.add(_conv(y, hid, 1, 1, 0, act="relu6"))
            y = b.add(_conv(y, hid, 3, stride, 1, groups=hid, act="relu6"))
            y = b.add(_conv(y, c, 1, 1, 0))
            if stride == 1 and cin == c:
                y = b.add({"type": "add", "in": [y, inp], "act": "none"})
            x = y
            cin = c
    x = b.add(_conv(x, 1280, 1, 1, 0, act="relu6"))
    x = b.add({"type": "gap", "in": [x]})
    b.add({"type": "fc", "in": [x], "k": 1000})
    return {"name": f"mobilenetv2_bs{batch}", "dtype": dtype, "batch": batch,
            "in_chw": [3, 224, 224], "input_dist": "uniform", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


VGG16_CONVS = [64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"]


def vgg16(batch=1, dtype="bf16", hw=224):
    """VGG16 shape: thirteen 3x3 convolutions with ReLU in five groups, each
    closed by 2x2/2 max pooling, then the classifier 4096 -> 4096 -> 1000.
    A straight chain (no branch or merge).  The first classifier layer reads
    the flattened 512 x (hw/32) x (hw/32) map; it is written as a convolution
    whose kernel covers that whole map (no padding), which is the same
    affine map on the NCHW-flattened input, so the net holds no reshape."""
    assert hw % 32 == 0, hw
    b = _Builder()
    x = 0
    for v in VGG16_CONVS:
        if v == "M":
            x = b.add({"type": "maxpool", "in": [x], "k": 2, "stride": 2, "pad": 0})
        else:
            x = b.add(_conv(x, v, 3, 1, 1, act="relu"))
    f = hw // 32
    x = b.add(_conv(x, 4096, f, 1, 0, act="relu"))
    x = b.add({"type": "fc", "in": [x], "k": 4096, "act": "relu"})
    b.add({"type": "fc", "in": [x], "k": 1000})
    return {"name": f"vgg16_bs{batch}_{dtype}" + ("" if hw == 224 else f"_{hw}px"), "dtype": dtype,
            "batch": batch, "in_chw": [3, hw, hw], "input_dist": "uniform", "seed": 0, "layers": b.layers,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


def net_d(batch=2, dtype="bf16"):
    """A two-input, two-output net (the multi-input/multi-output case of the
    auxiliary layers, Sec. IV-E): input 0 (3 x 20 x 20) and input 1
    (8 x 10 x 10) each pass a convolution, meet in an add, and the net ends
    in two heads -- a classifier after the merge and a map computed from the
    second input's branch."""
    L = [
        _conv(0, 16, 3, 2, 1, act="relu"),                    # 1: input 0 -> 16 x 10 x 10
        {"type": "input", "in": [], "chw": [8, 10, 10]},     # 2: input 1
        _conv(2, 16, 3, 1, 1, act="relu"),                    # 3: input 1 -> 16 x 10 x 10
        {"type": "add", "in": [1, 3], "act": "relu"},          # 4: merge
        _conv(4, 24, 3, 1, 1, act="relu"),                    # 5
        {"type": "gap", "in": [5]},                           # 6
        {"type": "fc", "in": [6], "k": 10},                   # 7: output 0
        _conv(3, 12, 1, 1, 0),                                # 8: output 1 (12 x 10 x 10)
    ]
    return {"name": f"net_d_bs{batch}_{dtype}", "dtype": dtype, "batch": batch, "in_chw": [3, 20, 20],
            "input_dist": "uniform", "seed": 0, "layers": L, "outputs": [7, 8],
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


def with_batch(spec, batch):
    out = copy.deepcopy(spec)
    out["batch"] = batch
    return out


def all_configs():
    """The five workloads: tiny chain, the conv sweep, ResNet-18, MobileNetV2, ResNet-50."""
    return {
        "tiny_chain": tiny_chain(),
        "conv_sweep": [conv_sweep(c, hw) for c, hw in CONV_SWEEP_SHAPES],
        "resnet18_bs1": resnet18(1),
        "mobilenetv2_bs1": mobilenet_v2(1),
        "mobilenetv2_bs8": mobilenet_v2(8),
        "resnet50_bs1_bf16": resnet50(1, "bf16"),
        "resnet50_bs32_bf16": resnet50(32, "bf16"),
        "resnet50_bs1_f16": resnet50(1, "f16"),
        "resnet50_bs32_f16": resnet50(32, "f16"),
    }


def edges(spec):
    """Edge list (j, i) of the layer DAG, layer 0 being the input (further
    input layers have no data edge)."""
    out = []
    for i, layer in enumerate(spec["layers"], start=1):
        for j in layer["in"]:
            out.append((j, i))
    return out


def channels(spec):
    """Channel count of every layer's output (index 0 = the input); structural only."""
    ch = [spec["in_chw"][0]]
    for layer in spec["layers"]:
        t = layer["type"]
        if t == "input":
            ch.append(layer["chw"][0])
        elif t in ("conv", "fc"):
            ch.append(layer["k"])
        else:
            ch.append(ch[layer["in"][0]])
    return ch


def fuse_residual(spec, tensors=None, only_1x1=True):
    """Structure-only transform: every residual add whose operand is a dense
    convolution without activation, consumed by that add alone (a 1x1 one if
    ``only_1x1``), becomes that convolution with the add's other operand as
    residual input and the add's activation, placed where the add was (all
    its inputs come earlier).  Returns the new spec and, if given, the
    generated tensors re-listed for the new layer order (no value changes)."""
    layers = spec["layers"]
    n = len(layers)
    consumers = {i: [] for i in range(n + 1)}
    for i, layer in enumerate(layers, start=1):
        for j in layer["in"]:
            consumers[j].append(i)
    fused_into = {}   # add id -> conv id
    for i, layer in enumerate(layers, start=1):
        if layer["type"] != "add":
            continue
        for a, b in ((layer["in"][0], layer["in"][1]), (layer["in"][1], layer["in"][0])):
            if a == 0:
                continue
            c = layers[a - 1]
            if (c["type"] == "conv" and len(c["in"]) == 1 and c["groups"] == 1 and c["act"] == "none"
                    and consumers[a] == [i] and a not in fused_into.values()
                    and (not only_1x1 or (c["r"] == 1 and c["s"] == 1))):
                fused_into[i] = a
                break
    gone = set(fused_into.values())
    order = []        # old ids in the new order; an add's slot takes its conv
    for i in range(1, n + 1):
        if i in gone:
            continue
        order.append(fused_into.get(i, i))
    new_id = {0: 0}
    for k, old in enumerate(order, start=1):
        new_id[old] = k
    for add_id, conv_id in fused_into.items():
        new_id[add_id] = new_id[conv_id]
    out_layers = []
    for old in order:
        lay = copy.deepcopy(layers[old - 1])
        add_id = next((a for a, c in fused_into.items() if c == old), None)
        if add_id is not None:
            add = layers[add_id - 1]
            other = add["in"][1] if add["in"][0] == old else add["in"][0]
            lay["in"] = [lay["in"][0], other]
            lay["act"] = add.get("act", "none")
        lay["in"] = [new_id[j] for j in lay["in"]]
        out_layers.append(lay)
    out = dict(spec, layers=out_layers, name=spec["name"] + "_fused")
    if tensors is None:
        return out
    t2 = dict(tensors, w=[tensors["w"][old - 1] for old in order], b=[tensors["b"][old - 1] for old in order])
    return out, t2

def fuse_projection(spec, tensors=None):
    """Structure-only transform, after ``fuse_residual``: a dense convolution
    whose residual input is a dense 1x1 convolution without padding,
    activation or residual of its own, consumed by it alone (the projection
    shortcut of a bottleneck block), takes that convolution's input as a
    projected shortcut (``"proj": {"stride": s}``): one layer computing
    act(conv(x) + b + conv1x1_s(shortcut) + b_proj).  The projection layer is
    removed; with ``tensors`` the fused layer's weights and biases become
    (own, projection) pairs.  Returns the new spec (and tensors)."""
    layers = spec["layers"]
    n = len(layers)
    consumers = {i: [] for i in range(n + 1)}
    for i, layer in enumerate(layers, start=1):
        for j in layer["in"]:
            consumers[j].append(i)
    fused = {}        # conv id -> projection id
    for i, layer in enumerate(layers, start=1):
        if layer["type"] != "conv" or len(layer["in"]) != 2 or layer.get("proj") or layer["groups"] != 1:
            continue
        p = layer["in"][1]
        if p == 0:
            continue
        pl = layers[p - 1]
        if (pl["type"] == "conv" and len(pl["in"]) == 1 and pl["groups"] == 1 and pl["act"] == "none"
                and pl["r"] == 1 and pl["s"] == 1 and pl["pad"] == 0 and not pl.get("proj")
                and consumers[p] == [i]):
            fused[i] = p
    gone = set(fused.values())
    order = [i for i in range(1, n + 1) if i not in gone]
    new_id = {0: 0}
    for k, old in enumerate(order, start=1):
        new_id[old] = k
    out_layers = []
    for old in order:
        lay = copy.deepcopy(layers[old - 1])
        if old in fused:
            pl = layers[fused[old] - 1]
            lay["in"] = [lay["in"][0], pl["in"][0]]
            lay["proj"] = {"stride": pl["stride"]}
        lay["in"] = [new_id[j] for j in lay["in"]]
        out_layers.append(lay)
    out = dict(spec, layers=out_layers, name=spec["name"] + "_proj")
    if "outputs" in spec:
        out["outputs"] = [new_id[o] for o in spec["outputs"]]
    if tensors is None:
        return out
    tw, tb = tensors["w"], tensors["b"]
    t2 = dict(tensors,
              w=[(tw[old - 1], tw[fused[old] - 1]) if old in fused else tw[old - 1] for old in order],
              b=[(tb[old - 1], tb[fused[old] - 1]) if old in fused else tb[old - 1] for old in order],
              inputs={new_id[k]: v for k, v in tensors.get("inputs", {}).items()})
    return out, t2


