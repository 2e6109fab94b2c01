"""Residual-add fusion (a residual add folded into the 1x1 convolution that
produces its operand): the spec transform, the oracle's fused layer, and the
library's routine sets and DPRS on fused graphs.  No GPU."""

import numpy as np
import pytest

from oracle import numeric as O
from oracle.select import blockwise, problem_from_costs
from paper_2110_06037_amd import build_from_spec
from tests.test_dprs_host import randomise
from workloads import fuse_projection, fuse_residual, generate, mobilenet_v2, resnet18, resnet50, weight_shapes


def _topological(spec):
    return all(j < i for i, layer in enumerate(spec["layers"], start=1) for j in layer["in"])


def mini_resnet():
    """Two bottleneck blocks (projection, then identity shortcut) on 1x16x8x8."""
    L = []
    def conv(i, k, r, st=1, act="none"):
        L.append({"type": "conv", "in": [i], "k": k, "r": r, "s": r, "stride": st, "pad": r // 2,
                  "groups": 1, "act": act})
        return len(L)
    x = conv(0, 16, 3, 1, "relu")
    for blk in range(2):
        inp = x
        y = conv(inp, 8, 1, act="relu")
        y = conv(y, 8, 3, act="relu")
        y = conv(y, 32, 1)
        sc = conv(inp, 32, 1) if blk == 0 else inp
        L.append({"type": "add", "in": [y, sc], "act": "relu"})
        x = len(L)
    L.append({"type": "gap", "in": [x]})
    L.append({"type": "fc", "in": [len(L)], "k": 10})
    return {"name": "mini_resnet", "dtype": "bf16", "batch": 2, "in_chw": [16, 8, 8],
            "input_dist": "uniform", "seed": 0, "layers": L,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


def test_resnet50_every_bottleneck_add_is_fused():
    spec = resnet50(1)
    fused = fuse_residual(spec)
    n_add = sum(l["type"] == "add" for l in spec["layers"])
    assert n_add == 16
    assert len(fused["layers"]) == len(spec["layers"]) - 16
    assert not any(l["type"] == "add" for l in fused["layers"])
    res = [l for l in fused["layers"] if l["type"] == "conv" and len(l["in"]) == 2]
    assert len(res) == 16 and all(l["r"] == 1 and l["act"] == "relu" for l in res)
    assert _topological(fused)
    assert weight_shapes(fused).count(None) == weight_shapes(spec).count(None) - 16


def test_mobilenet_projection_adds_are_fused_and_resnet18_shortcut_projections():
    mb = mobilenet_v2(1)
    fused = fuse_residual(mb)
    n_add = sum(l["type"] == "add" for l in mb["layers"])
    assert n_add == 10 and not any(l["type"] == "add" for l in fused["layers"])
    assert all(l["act"] == "none" for l in fused["layers"] if len(l["in"]) == 2)
    # ResNet-18: identity-shortcut adds follow 3x3 convolutions (left alone by the
    # 1x1 rule); the three projection-shortcut adds fold into the 1x1 projection
    r18 = resnet18(1)
    f18 = fuse_residual(r18)
    assert sum(l["type"] == "add" for l in f18["layers"]) == 5
    res = [l for l in f18["layers"] if len(l["in"]) == 2 and l["type"] == "conv"]
    assert len(res) == 3 and all(l["r"] == 1 and l["stride"] == 2 and l["act"] == "relu" for l in res)
    assert _topological(f18)


def test_fused_net_computes_the_unfused_net():
    # exact arithmetic (no storage rounding): the transform only moves layers
    # and weights, so both nets give the same outputs up to fp64 rounding
    spec = mini_resnet()
    t = generate(spec)
    fused, tf = fuse_residual(spec, t)
    assert len(fused["layers"]) == len(spec["layers"]) - 2 and _topological(fused)
    from workloads import to_f64
    dec = lambda tens: {"x": to_f64(tens["x"], spec["dtype"]),
                        "w": [None if w is None else to_f64(w, spec["dtype"]) for w in tens["w"]],
                        "b": [None if b is None else b.astype(np.float64) for b in tens["b"]]}
    a = O.forward(spec, dec(t), storage="fp64")[-1]
    b = O.forward(fused, dec(tf), storage="fp64")[-1]
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    # with storage rounding the fused net rounds once where the unfused rounds twice
    a = O.forward(spec, dec(t))[-1]
    b = O.forward(fused, dec(tf))[-1]
    assert np.linalg.norm(a - b) / np.linalg.norm(a) < 2e-2


def test_fused_graph_routines_and_dprs():
    spec = fuse_residual(resnet50(1))
    g = build_from_spec(spec, device=-1)
    for i, layer in enumerate(spec["layers"], start=1):
        if layer["type"] == "conv" and len(layer["in"]) == 2:
            names = [r["name"] for r in g.routines(i)]
            assert names and not any("winograd" in n for n in names)
    costs = randomise(g.costs(), 77, max_cost=100)
    g.set_costs(costs)
    g.select("dprs")
    ids, total = g.path()
    t, tup = blockwise(problem_from_costs(costs), [0, 1, 2])
    assert tuple(ids) + (0,) == tup and total == t
    g.close()


def test_resnet50_projection_shortcuts_fold_into_the_expand_convolutions():
    fused = fuse_residual(resnet50(1))
    proj = fuse_projection(fused)
    assert len(proj["layers"]) == len(fused["layers"]) - 4 and _topological(proj)
    pl = [(i, l) for i, l in enumerate(proj["layers"], start=1) if l.get("proj")]
    assert [l["proj"]["stride"] for _, l in pl] == [1, 2, 2, 2]
    for i, l in pl:
        # the main input is the block's last 1x1 reduce path, the shortcut
        # the block input (the previous stage's output), both earlier layers
        assert l["type"] == "conv" and l["r"] == 1 and l["act"] == "relu" and len(l["in"]) == 2
        assert l["in"][1] < l["in"][0] < i
    # nothing to fold where the projection is not a lone 1x1 residual operand
    assert len(fuse_projection(fuse_residual(resnet18(1)))["layers"]) == len(fuse_residual(resnet18(1))["layers"])
    assert len(fuse_projection(fuse_residual(mobilenet_v2(1)))["layers"]) == \
        len(fuse_residual(mobilenet_v2(1))["layers"])


def test_projection_fused_net_computes_the_unfused_net():
    # mini_resnet's first block has a projection shortcut: after both folds
    # one layer computes conv + projection; exact arithmetic gives the same
    # outputs, storage rounding differs only by the rounding the fold removes
    from workloads import decode
    spec = mini_resnet()
    t = generate(spec)
    fused, tf = fuse_residual(spec, t)
    proj, tp = fuse_projection(fused, tf)
    assert len(proj["layers"]) == len(spec["layers"]) - 3 and _topological(proj)
    assert sum(bool(l.get("proj")) for l in proj["layers"]) == 1
    a = O.forward(spec, decode(t, "bf16"), storage="fp64")[-1]
    b = O.forward(proj, decode(tp, "bf16"), storage="fp64")[-1]
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    a = O.forward(spec, decode(t, "bf16"))[-1]
    b = O.forward(proj, decode(tp, "bf16"))[-1]
    assert np.linalg.norm(a - b) / np.linalg.norm(a) < 2e-2


def test_projected_layers_routines_and_dprs():
    spec = fuse_projection(fuse_residual(resnet50(1)))
    g = build_from_spec(spec, device=-1)
    for i, layer in enumerate(spec["layers"], start=1):
        if layer.get("proj"):
            rts = g.routines(i)
            # the two-launch direct routine in every layout, the one-kernel
            # implicit GEMM in the channel-vector layouts only
            assert {r["layout"] for r in rts if r["algo"] == 0} == {0, 1, 2}
            assert {r["layout"] for r in rts if r["algo"] == 1} == {1, 2}
            assert not any(r["algo"] == 2 for r in rts)
    costs = randomise(g.costs(), 91, max_cost=100)
    g.set_costs(costs)
    g.select("dprs")
    ids, total = g.path()
    t, tup = blockwise(problem_from_costs(costs), [0, 1, 2])
    assert tuple(ids) + (0,) == tup and total == t
    g.close()
