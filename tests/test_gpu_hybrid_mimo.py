"""GPU parity of precision-hybrid paths and multi-input/multi-output nets.

Hybrid (Sec. IV-F): schemas are (dtype, layout) pairs; a path may compute
its layers in float32, float16 and bfloat16, with cast adapts between them.
The oracle of such a path is the chained float64 forward pass in which each
layer reads its inputs cast to its own dtype, uses the weights rounded to it
and stores its output rounded to it.  Multi-input/multi-output nets
(Sec. IV-E) run through sn_run_mimo and are compared output by output."""

import numpy as np
import pytest

from oracle import numeric as O
from oracle.select import exhaustive, problem_from_costs
from paper_2110_06037_amd import Graph, build_from_spec, native as N
from tests.gpu_util import TOL, err, from_dev, to_dev
from tests.test_fusion_host import mini_resnet
from workloads import generate, net_d, random_tensor, tiny_chain, to_f64

pytestmark = pytest.mark.gpu

DT = {0: "f32", 1: "f16", 2: "bf16"}


def decoded(spec, t):
    dt = spec["dtype"]
    return {"x": to_f64(t["x"], dt), "w": [None if w is None else to_f64(w, dt) for w in t["w"]],
            "b": [None if b is None else b.astype(np.float64) for b in t["b"]],
            "inputs": {k: to_f64(v, dt) for k, v in t.get("inputs", {}).items()}}


def path_dtypes(g, spec):
    ids = g.path()[0]
    return [spec["dtype"]] + [DT[g.routines(i)[ids[i]]["dtype"]] for i in range(1, len(ids))]


def tol_for(ldt):
    return TOL["f32"] if all(d == "f32" for d in ldt[1:]) else TOL["bf16"]


def check_path(g, spec, t):
    import torch
    ldt = path_dtypes(g, spec)
    ref = O.forward(spec, decoded(spec, t), storage="dtype", layer_dtypes=ldt)[-1]
    y = g.run(to_dev(t["x"], spec["dtype"]))
    torch.cuda.synchronize()
    got = from_dev(y, spec["dtype"]).reshape(spec["batch"], -1)
    e = err(got, ref.reshape(spec["batch"], -1), "f32" if tol_for(ldt) == TOL["f32"] else "bf16")
    return e, tol_for(ldt), ldt


@pytest.mark.parametrize("io,shape", [("f32", (2, 5, 9, 7)), ("bf16", (1, 16, 6, 6)), ("f16", (3, 8, 5, 4))])
def test_cast_converters_bit_exact(io, shape):
    # an identity layer (1x1 max pooling) in every schema: the input is cast
    # and converted into it and back into the run dtype's NCHW output; the
    # stored intermediate must be the one rounding of the input to the
    # schema's dtype, in its layout, with zero-padded NC8HW8 channels
    import torch
    n, c, h, w = shape
    x = random_tensor(shape, io, seed=3, dist="normal", scale=3.0)
    x64 = to_f64(x, io)
    g = Graph(io, n, c, h, w, device=0, dtypes=["f32", "f16", "bf16"])
    g.add_maxpool(0, 1, 1, 0)
    g.set_option(N.OPT_KEEP, 1)
    xd = to_dev(x, io)
    for rt in g.routines(1):
        g.set_path([0, rt["id"]])
        y = g.run(xd)
        torch.cuda.synchronize()
        d = DT[rt["dtype"]]
        mid = O.round_to(x64, d)
        want = O.round_to(mid, io)
        assert np.array_equal(from_dev(y, io).reshape(shape), want), rt["name"]
        if DT[rt["dtype"]] == io and rt["layout"] == N.NCHW:
            continue                          # stored straight into the caller's output
        buf, lay = g.layer_output(1)
        torch.cuda.synchronize()
        raw = buf.cpu().numpy()
        vals = raw.view(np.float32) if d == "f32" else raw.view(np.uint16)
        if lay == N.NCHW:
            v = vals.reshape(n, c, h, w)
        elif lay == N.NHWC:
            v = vals.reshape(n, h, w, c).transpose(0, 3, 1, 2)
        else:
            c8 = (c + 7) // 8 * 8
            v = vals.reshape(n, c8 // 8, h, w, 8).transpose(0, 1, 4, 2, 3).reshape(n, c8, h, w)
            assert not np.any(v[:, c:]), rt["name"]
            v = v[:, :c]
        got = v.astype(np.float64) if d == "f32" else to_f64(v if d == "bf16" else v.view(np.float16), d)
        assert np.array_equal(got, mid), rt["name"]
    g.close()


@pytest.mark.parametrize("name,io", [("tiny", "f32"), ("mini_resnet", "bf16"), ("mini_resnet", "f32")])
def test_hybrid_dprs_on_the_measured_table(name, io):
    # all three dtypes allowed: DPRS on the measured table equals the
    # exhaustive optimum (tiny net), and the selected (possibly mixed) path
    # matches the oracle of its per-layer dtypes
    spec = dict(tiny_chain() if name == "tiny" else mini_resnet(), dtype=io)
    t = generate(spec)
    kw = dict(layouts=["NCHW", "NHWC"], algos=["igemm"], params=False) if name == "tiny" else {}
    g = build_from_spec(spec, t, dtypes=["f32", "f16", "bf16"], **kw)
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    if name == "tiny":
        tt, tup, _ = exhaustive(problem_from_costs(g.costs()))
        ids, total = g.path()
        assert tuple(ids) + (0,) == tup and total == tt
    e, tol, ldt = check_path(g, spec, t)
    print(f"{name} {io} hybrid dprs dtypes {ldt} err {e:.2e}", flush=True)
    assert e <= tol
    g.close()


@pytest.mark.parametrize("io", ["bf16", "f32"])
def test_forced_mixed_precision_path(io):
    # every layer in the next dtype of (bf16, f32, f16) and the next layout:
    # a cast adapt (often with a layout change) on every edge
    spec = dict(mini_resnet(), dtype=io)
    t = generate(spec)
    g = build_from_spec(spec, t, dtypes=["f32", "f16", "bf16"])
    cyc = [2, 0, 1]
    ids = [0]
    for i in range(1, g.num_layers()):
        rts = g.routines(i)
        want = [r for r in rts if r["dtype"] == cyc[i % 3] and r["layout"] == i % 3] or \
               [r for r in rts if r["dtype"] == cyc[i % 3]]
        ids.append(min(want, key=lambda r: (r["algo"] != 1, r["id"]))["id"])
    g.set_path(ids)
    ldt = path_dtypes(g, spec)
    assert len(set(ldt[1:])) == 3
    e, tol, _ = check_path(g, spec, t)
    print(f"forced mixed path {io}: {ldt} err {e:.2e}", flush=True)
    assert e <= tol
    # the same path with every intermediate kept, timed repetition included
    import torch
    xd = to_dev(t["x"], io)
    y0 = g.run(xd)
    torch.cuda.synchronize()
    y1, ms = g.run_timed(xd, reps=3)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(y0, io), from_dev(y1, io))
    g.close()


def _mimo_out(g, spec, t):
    import torch
    xs = [to_dev(t["x"], spec["dtype"])] + [to_dev(t["inputs"][k], spec["dtype"]) for k in sorted(t["inputs"])]
    outs = g.run_mimo(xs, output_layers=spec["outputs"])
    torch.cuda.synchronize()
    return [from_dev(o, spec["dtype"]).reshape(spec["batch"], -1) for o in outs], xs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_two_input_two_output_net(dtype):
    spec = net_d(3, dtype)
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    refs = O.forward(spec, decoded(spec, t), storage="dtype")
    refs = [refs[o].reshape(spec["batch"], -1) for o in spec["outputs"]]
    g.select("dprs")
    with pytest.raises(N.SNError):
        g.run(to_dev(t["x"], dtype))          # a two-input net needs sn_run_mimo
    outs, xs = _mimo_out(g, spec, t)
    for k, (o, r) in enumerate(zip(outs, refs)):
        e = err(o, r, dtype)
        print(f"net D {dtype} dprs output {k} err {e:.2e}", flush=True)
        assert e <= TOL[dtype], k
    for lay in ("NCHW", "NHWC", "NC8HW8"):
        for algo in ("igemm", "winograd", "direct"):
            g.select("fixed", lay, algo)
            outs, _ = _mimo_out(g, spec, t)
            for k, (o, r) in enumerate(zip(outs, refs)):
                assert err(o, r, dtype) <= TOL[dtype], (lay, algo, k)
    # integrated profiling and HIP-graph replay of a multi-output plan
    g.profile_integrated(warmup=1, reps=2)
    eager, _ = _mimo_out(g, spec, t)
    g.set_option(N.OPT_HIPGRAPH, 1)
    for rep in range(3):
        outs, _ = _mimo_out(g, spec, t)
        for a, b in zip(outs, eager):
            assert np.array_equal(a, b), rep
    g.close()


def test_mimo_with_hybrid_dtypes():
    spec = net_d(2, "f32")
    t = generate(spec)
    g = build_from_spec(spec, t, dtypes=["f32", "f16", "bf16"])
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    ldt = path_dtypes(g, spec)
    refs = O.forward(spec, decoded(spec, t), storage="dtype", layer_dtypes=ldt)
    outs, _ = _mimo_out(g, spec, t)
    tol = tol_for(ldt)
    for k, o in enumerate(spec["outputs"]):
        e = err(outs[k], refs[o].reshape(spec["batch"], -1), "f32" if tol == TOL["f32"] else "bf16")
        print(f"net D hybrid {ldt} output {k} err {e:.2e}", flush=True)
        assert e <= tol
    g.close()
