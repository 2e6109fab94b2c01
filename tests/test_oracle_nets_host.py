"""Pins of the oracle's whole-net forward pass on branching nets.

``oracle.numeric.forward`` walks a layer DAG: residual adds, projection
shortcuts, convolutions with a folded residual input, depthwise layers and a
linear bottleneck.  Here it is checked against an independent evaluation of
the same nets written with torch's float64 functional operators (a library
convolution, pooling and matrix product), so a wrong input index, a dropped
shortcut, an activation in the wrong place or a residual added after instead
of before the activation fails.  No GPU."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import numeric as O
from tests.test_fusion_host import mini_resnet
from workloads import fuse_residual, generate, mobilenet_v2, resnet18, to_f64, with_batch


def _act(t, act):
    if act == "relu":
        return torch.clamp(t, min=0.0)
    if act == "relu6":
        return torch.clamp(t, 0.0, 6.0)
    assert act == "none"
    return t


def torch_forward(spec, t, round_f32=False):
    """Every layer output of the net, evaluated with torch float64 ops;
    round_f32 rounds each layer output to float32 (one rounding)."""
    dt = spec["dtype"]
    outs = [torch.from_numpy(to_f64(t["x"], dt))]
    for i, L in enumerate(spec["layers"]):
        ins = [outs[j] for j in L["in"]]
        w = None if t["w"][i] is None else torch.from_numpy(to_f64(t["w"][i], dt))
        b = None if t["b"][i] is None else torch.from_numpy(t["b"][i].astype(np.float64))
        kind = L["type"]
        if kind == "conv":
            y = F.conv2d(ins[0], w, b, stride=L["stride"], padding=L["pad"], groups=L["groups"])
            if len(ins) == 2:
                y = y + ins[1]
            y = _act(y, L["act"])
        elif kind == "maxpool":
            y = F.max_pool2d(ins[0], L["k"], L["stride"], L["pad"])
        elif kind == "gap":
            y = ins[0].mean(dim=(2, 3), keepdim=True)
        elif kind == "add":
            y = _act(ins[0] + ins[1], L.get("act", "none"))
        elif kind == "fc":
            n = ins[0].shape[0]
            y = _act(F.linear(ins[0].reshape(n, -1), w, b), L.get("act", "none")).reshape(n, -1, 1, 1)
        else:
            raise ValueError(kind)
        if round_f32:
            y = y.to(torch.float32).to(torch.float64)
        outs.append(y)
    return [o.numpy() for o in outs]


def inverted_residual_net():
    """A MobileNetV2-style piece on 2x8x12x10: stem, an inverted-residual block
    with a stride-1 depthwise layer, a linear 1x1 bottleneck and an identity
    shortcut, then a stride-2 block (no shortcut), gap and FC."""
    L = []

    def conv(i, k, r, st=1, groups=1, act="none"):
        L.append({"type": "conv", "in": [i], "k": k, "r": r, "s": r, "stride": st, "pad": r // 2,
                  "groups": groups, "act": act})
        return len(L)

    x = conv(0, 16, 3, 1, act="relu6")
    y = conv(x, 96, 1, act="relu6")
    y = conv(y, 96, 3, 1, groups=96, act="relu6")
    y = conv(y, 16, 1)
    L.append({"type": "add", "in": [y, x], "act": "none"})
    x = len(L)
    y = conv(x, 48, 1, act="relu6")
    y = conv(y, 48, 3, 2, groups=48, act="relu6")
    y = conv(y, 24, 1)
    L.append({"type": "gap", "in": [y]})
    L.append({"type": "fc", "in": [len(L)], "k": 7})
    return {"name": "inverted_residual", "dtype": "bf16", "batch": 2, "in_chw": [8, 12, 10],
            "input_dist": "uniform", "seed": 3, "layers": L,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


def resnet18_first_stages():
    """ResNet-18 at 2x3x40x40 cut after its first two stages: basic blocks with
    identity shortcuts and a stride-2 block with a 1x1 projection."""
    spec = resnet18(2)
    keep = []
    for L in spec["layers"]:
        keep.append(L)
        if L["type"] == "add" and sum(l["type"] == "add" for l in keep) == 4:
            break
    n = len(keep)
    keep.append({"type": "gap", "in": [n]})
    keep.append({"type": "fc", "in": [n + 1], "k": 5})
    return dict(spec, name="resnet18_2stages", in_chw=[3, 40, 40], layers=keep)


NETS = {
    "mini_resnet": mini_resnet,
    "mini_resnet_fused": lambda: fuse_residual(mini_resnet()),
    "inverted_residual": inverted_residual_net,
    "inverted_residual_fused": lambda: fuse_residual(inverted_residual_net()),
    "resnet18_2stages": resnet18_first_stages,
    "resnet18_2stages_fused": lambda: fuse_residual(resnet18_first_stages()),
}


@pytest.mark.parametrize("name", sorted(NETS))
def test_forward_on_branching_nets_matches_torch_f64(name):
    spec = NETS[name]()
    assert any(len(L["in"]) == 2 for L in spec["layers"]), "the net must merge branches"
    t = generate(spec)
    dt = spec["dtype"]
    dec = {"x": to_f64(t["x"], dt), "w": [None if w is None else to_f64(w, dt) for w in t["w"]],
           "b": [None if b is None else b.astype(np.float64) for b in t["b"]]}
    ours = O.forward(spec, dec, storage="f64", keep=True)
    ref = torch_forward(spec, t)
    assert len(ours) == len(ref)
    for i, (a, b) in enumerate(zip(ours, ref)):
        a = a.reshape(b.shape)
        scale = max(np.max(np.abs(b)), 1e-30)
        assert np.max(np.abs(a - b)) / scale <= 1e-12, (name, i)


@pytest.mark.parametrize("name", ["mini_resnet", "inverted_residual_fused"])
def test_forward_storage_rounding_matches_torch_per_layer_f32(name):
    # storage="dtype" in float32 rounds every layer output once, as torch's
    # float64 -> float32 conversion does
    spec = dict(NETS[name](), dtype="f32")
    t = generate(spec)
    dec = {"x": to_f64(t["x"], "f32"), "w": [None if w is None else to_f64(w, "f32") for w in t["w"]],
           "b": [None if b is None else b.astype(np.float64) for b in t["b"]]}
    ours = O.forward(spec, dec, storage="dtype", keep=True)
    ref = torch_forward(spec, t, round_f32=True)
    for i, (a, b) in enumerate(zip(ours[1:], ref[1:]), start=1):
        a = a.reshape(b.shape)
        scale = max(np.max(np.abs(b)), 1e-30)
        # the two sides sum in different orders before the one rounding
        assert np.max(np.abs(a - b)) / scale <= 2 ** -22, (name, i)


def test_forward_on_image_subsets_equals_the_batch():
    # the sampled-image checks of the GPU tests run the oracle on a subset of
    # the batch: images are independent, so rows of the full-batch output
    spec = with_batch(inverted_residual_net(), 4)
    t = generate(spec)
    dec = {"x": to_f64(t["x"], "bf16"), "w": [None if w is None else to_f64(w, "bf16") for w in t["w"]],
           "b": [None if b is None else b.astype(np.float64) for b in t["b"]]}
    full = O.forward(spec, dec)[-1]
    pick = [3, 1]
    sub = dict(dec, x=dec["x"][pick])
    part = O.forward(with_batch(spec, len(pick)), sub)[-1]
    assert np.array_equal(part, full[pick])


def test_mobilenet_v2_block_structure_is_what_the_pin_covers():
    # the real MobileNetV2 spec has the linear bottleneck (no activation on
    # the projection) and identity adds without activation, as the pin net
    spec = mobilenet_v2(1)
    adds = [L for L in spec["layers"] if L["type"] == "add"]
    assert adds and all(L["act"] == "none" for L in adds)
    for L in adds:
        proj = spec["layers"][L["in"][0] - 1]
        assert proj["type"] == "conv" and proj["r"] == 1 and proj["act"] == "none"
