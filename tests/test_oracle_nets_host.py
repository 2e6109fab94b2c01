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
from workloads import (decode, fuse_projection, fuse_residual, generate, materialise, mobilenet_v2, net_d, resnet18,
                       resnet50, to_f64, with_batch)


def _act(t, act):
    if act == "relu":
        return torch.clamp(t, min=0.0)
    if act == "relu6":
        return torch.clamp(t, 0.0, 6.0)
    assert act == "none"
    return t


def _round(a, dtype):
    """One rounding of float64 values to dtype, by the input generator's
    conversion (numpy's half cast, the generator's bfloat16 rounding)."""
    return torch.from_numpy(to_f64(materialise(a.numpy(), dtype), dtype))


def torch_forward(spec, t, round_f32=False, layer_dtypes=None):
    """Every layer output of the net, evaluated with torch float64 ops;
    round_f32 rounds each layer output to float32 (one rounding);
    layer_dtypes (indexed by layer id) casts a layer's inputs and weights to
    its dtype and rounds its output to it, and casts the net outputs back."""
    dt = spec["dtype"]
    outs = [torch.from_numpy(to_f64(t["x"], dt))]
    ldt = layer_dtypes or [dt] * (len(spec["layers"]) + 1)
    for i, L in enumerate(spec["layers"]):
        if L["type"] == "input":
            outs.append(torch.from_numpy(to_f64(t["inputs"][i + 1], dt)))
            continue
        me = ldt[i + 1]

        def src_dtype(j):  # inputs carry the spec's dtype
            return dt if j == 0 or spec["layers"][j - 1]["type"] == "input" else ldt[j]

        ins = [outs[j] if layer_dtypes is None or src_dtype(j) == me else _round(outs[j], me) for j in L["in"]]
        if L.get("proj"):
            # a projected shortcut: torch's convolution of each input with its
            # own weights and bias, summed, then the activation
            (w1, w2), (b1, b2) = t["w"][i], t["b"][i]
            ws_ = [torch.from_numpy(to_f64(v, dt)) for v in (w1, w2)]
            if me != dt:
                ws_ = [_round(v, me) for v in ws_]
            y = F.conv2d(ins[0], ws_[0], torch.from_numpy(b1.astype(np.float64)), stride=L["stride"],
                         padding=L["pad"])
            y = y + F.conv2d(ins[1], ws_[1], torch.from_numpy(b2.astype(np.float64)), stride=L["proj"]["stride"])
            y = _act(y, L["act"])
            if round_f32:
                y = y.to(torch.float32).to(torch.float64)
            if layer_dtypes is not None:
                y = _round(y, me)
            outs.append(y)
            continue
        w = None if t["w"][i] is None else torch.from_numpy(to_f64(t["w"][i], dt))
        if w is not None and me != dt:
            w = _round(w, me)
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
        if layer_dtypes is not None:
            y = _round(y, me)
        outs.append(y)
    if layer_dtypes is not None:
        for o in spec.get("outputs", [len(spec["layers"])]):
            if ldt[o] != dt:
                outs[o] = _round(outs[o], dt)
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


def resnet50_first_stages():
    """ResNet-50 at 2x3x48x48 cut after its second stage's first block: the
    stem, stage 1 (a projection shortcut at stride 1, identity shortcuts) and
    a stride-2 projection block."""
    spec = resnet50(2)
    keep = []
    for L in spec["layers"]:
        keep.append(L)
        if L["type"] == "add" and sum(l["type"] == "add" for l in keep) == 4:
            break
    n = len(keep)
    keep.append({"type": "gap", "in": [n]})
    keep.append({"type": "fc", "in": [n + 1], "k": 5})
    return dict(spec, name="resnet50_2stages", in_chw=[3, 48, 48], layers=keep)


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
    "mini_resnet_proj": lambda: fuse_projection(fuse_residual(mini_resnet())),
    "resnet50_2stages_proj": lambda: fuse_projection(fuse_residual(resnet50_first_stages())),
}


@pytest.mark.parametrize("name", sorted(NETS))
def test_forward_on_branching_nets_matches_torch_f64(name):
    spec = NETS[name]()
    assert any(len(L["in"]) == 2 for L in spec["layers"]), "the net must merge branches"
    t = generate(spec)
    dt = spec["dtype"]
    ours = O.forward(spec, decode(t, dt), storage="f64", keep=True)
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


def _decoded(spec, t):
    return decode(t, spec["dtype"])


def test_forward_on_a_two_input_two_output_net_matches_torch_f64():
    # further input layers take the caller's tensor; both outputs are kept
    spec = net_d()
    t = generate(spec)
    assert set(t["inputs"]) == {2}
    ours = O.forward(spec, _decoded(spec, t), storage="f64")
    ref = torch_forward(spec, t)
    for o in spec["outputs"]:
        assert ours[o] is not None
        a, b = ours[o].reshape(ref[o].shape), ref[o]
        assert np.max(np.abs(a - b)) / np.max(np.abs(b)) <= 1e-12, o


ULP = {"f32": 2.0 ** -23, "f16": 2.0 ** -10, "bf16": 2.0 ** -7}


@pytest.mark.parametrize("io", ["bf16", "f32"])
@pytest.mark.parametrize("name", ["inverted_residual", "mini_resnet_fused", "mini_resnet_proj", "net_d"])
def test_forward_with_per_layer_dtypes_matches_torch(name, io):
    # a precision-hybrid path: layer dtypes cycle through bf16, f32, f16; the
    # oracle and the torch evaluation cast inputs and weights at the same
    # places, so every layer output agrees to within one unit in the last
    # place of its dtype (the two sums differ only in order before the one
    # rounding), and almost all elements agree exactly
    # (float32 tensors at the ends make the weight casts round)
    spec = dict(net_d() if name == "net_d" else NETS[name](), dtype=io)
    t = generate(spec)
    cyc = ["bf16", "f32", "f16"]
    ldt = [spec["dtype"]] + [cyc[i % 3] for i in range(len(spec["layers"]))]
    ours = O.forward(spec, _decoded(spec, t), storage="dtype", keep=True, layer_dtypes=ldt)
    ref = torch_forward(spec, t, layer_dtypes=ldt)
    same = total = 0
    for i in range(1, len(ref)):
        if spec["layers"][i - 1]["type"] == "input":
            continue
        a, b = ours[i].reshape(ref[i].shape), ref[i]
        outs = spec.get("outputs", [len(spec["layers"])])
        d = spec["dtype"] if i in outs else ldt[i]
        tol = np.maximum(np.abs(b), 2.0 ** -14) * 2 * ULP[d]
        assert np.all(np.abs(a - b) <= tol), (name, i)
        same += int(np.sum(a == b))
        total += a.size
    assert same >= 0.99 * total, (same, total)
