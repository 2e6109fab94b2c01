"""Whole-net parity on the GPU: the DPRS-selected path and the fixed paths of
the synthetic workloads against the chained float64 oracle (every layer
output rounded to the run dtype), the DP path on the measured cost table
against exhaustive enumeration, full-size sampled checks at the benchmark's
shapes, and HIP-graph replay."""

import numpy as np
import pytest

from oracle import numeric as O
from oracle.select import blockwise, exhaustive, problem_from_costs
from paper_2110_06037_amd import build_from_spec, native as N
from tests.gpu_util import TOL, err, from_dev, to_dev
from workloads import (CONV_SWEEP_SHAPES, conv_sweep, fuse_residual, generate, mobilenet_v2, resnet18, resnet50,
                       tiny_chain, to_f64, vgg16, with_batch)

pytestmark = pytest.mark.gpu


def decoded(t, dtype):
    return {"x": to_f64(t["x"], dtype),
            "w": [None if w is None else to_f64(w, dtype) for w in t["w"]],
            "b": [None if b is None else b.astype(np.float64) for b in t["b"]]}


def oracle_out(spec, t, images=None):
    d = decoded(t, spec["dtype"])
    s = spec
    if images is not None:
        d["x"] = d["x"][:images]
        s = with_batch(spec, images)
    out = O.forward(s, d, storage="dtype")[-1]
    return out.reshape(out.shape[0], -1)


def run_out(g, spec, t):
    import torch
    xd = to_dev(t["x"], spec["dtype"])
    y = g.run(xd)
    torch.cuda.synchronize()
    return from_dev(y, spec["dtype"]).reshape(spec["batch"], -1), xd


def test_tiny_chain_measured_table_dp_equals_exhaustive_and_parity():
    spec = tiny_chain()
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=3, reps=10)
    costs = g.costs()
    for l in costs["layers"][1:-1]:
        assert all(r["ns"] > 0 for r in l["routines"]), l
    g.select("dprs")
    ids, total = g.path()
    tt, tup, count = exhaustive(problem_from_costs(costs))
    assert tuple(ids) + (0,) == tup and total == tt
    ref = oracle_out(spec, t)
    out, xd = run_out(g, spec, t)
    assert err(out, ref, "f32") <= TOL["f32"]
    # the timed run repeats every layer's launches; its result is the same bits
    y, ms = g.run_timed(xd, reps=3)
    assert np.array_equal(from_dev(y, "f32").reshape(spec["batch"], -1), out)
    assert ms[0] == 0 and all(m > 0 for m in ms[1:]), ms
    # cache-cold timing: a scratch buffer is written before each layer; the
    # result is unchanged
    g.set_option(N.OPT_FLUSH, 64 << 20)
    y, ms = g.run_timed(xd, reps=1)
    g.set_option(N.OPT_FLUSH, 0)
    assert np.array_equal(from_dev(y, "f32").reshape(spec["batch"], -1), out)
    assert ms[0] == 0 and all(m > 0 for m in ms[1:]), ms
    for lay in ("NCHW", "NHWC"):
        for algo in ("direct", "igemm"):
            g.select("fixed", lay, algo)
            out, _ = run_out(g, spec, t)
            assert err(out, ref, "f32") <= TOL["f32"], (lay, algo)


@pytest.mark.parametrize("name", ["tiny", "mobilenetv2"])
def test_integrated_profiling_selects_the_measured_fastest_candidate(name):
    spec = tiny_chain() if name == "tiny" else mobilenet_v2(1)
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    dp_ids, dp_t = g.path()
    cands = g.profile_integrated(warmup=2, reps=5)
    print(name, [(c["kind"], c["a"], c["b"], c["model_ns"], c["measured_ns"]) for c in cands],
          flush=True)
    assert cands[0]["kind"] == "dprs" and cands[0]["path"] == dp_ids and cands[0]["model_ns"] == dp_t
    assert all(c["measured_ns"] > 0 for c in cands)
    best = min(range(len(cands)), key=lambda i: (cands[i]["measured_ns"], i))
    ids, total = g.path()
    assert ids == cands[best]["path"] and total == cands[best]["model_ns"]
    out, _ = run_out(g, spec, t)
    assert err(out, oracle_out(spec, t), spec["dtype"]) <= TOL[spec["dtype"]]
    g.close()


@pytest.mark.parametrize("name", ["resnet18", "mobilenetv2", "resnet50_bf16", "resnet50_f16",
                                  "resnet50_fused", "mobilenetv2_fused", "vgg16_64px"])
def test_net_dp_and_fixed_paths_match_oracle(name):
    spec = {"resnet18": lambda: resnet18(1), "mobilenetv2": lambda: mobilenet_v2(1),
            "vgg16_64px": lambda: vgg16(2, "bf16", 64),
            "resnet50_bf16": lambda: resnet50(1, "bf16"),
            "resnet50_f16": lambda: resnet50(1, "f16"),
            "resnet50_fused": lambda: fuse_residual(resnet50(1, "bf16")),
            "mobilenetv2_fused": lambda: fuse_residual(mobilenet_v2(1))}[name]()
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    ref = oracle_out(spec, t)
    g.select("dprs")
    out, _ = run_out(g, spec, t)
    e = err(out, ref, spec["dtype"])
    print(f"{name} dprs err {e:.3e}", flush=True)
    assert e <= TOL[spec["dtype"]]
    costs = g.costs()
    tt, tup = blockwise(problem_from_costs(costs), [0, 1, 2])
    assert tuple(g.path()[0]) + (0,) == tup and g.path()[1] == tt
    for lay in ("NCHW", "NHWC", "NC8HW8"):
        for algo in ("igemm", "winograd", "direct"):
            g.select("fixed", lay, algo)
            out, _ = run_out(g, spec, t)
            e = err(out, ref, spec["dtype"])
            print(f"{name} fixed {lay}/{algo} err {e:.3e}", flush=True)
            assert e <= TOL[spec["dtype"]], (lay, algo)
    g.close()


def test_resnet50_bs32_dp_path_sampled_images():
    # the benchmark's configuration: full batch on the GPU, images 0 and 1
    # through the oracle (images are independent)
    spec = resnet50(32, "bf16")
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    out, _ = run_out(g, spec, t)
    ref = oracle_out(spec, t, images=2)
    e = err(out[:2], ref, "bf16")
    print(f"resnet50 bs32 dprs images 0-1 err {e:.3e}", flush=True)
    assert e <= TOL["bf16"]
    assert np.all(np.isfinite(out))
    g.close()


@pytest.mark.parametrize("si", range(len(CONV_SWEEP_SHAPES)))
def test_conv_sweep_full_size_sampled(si):
    # full-size layer (batch 32, fp16): every routine checked on 3000 sampled outputs
    c, hw = CONV_SWEEP_SHAPES[si]
    spec = conv_sweep(c, hw)
    t = generate(spec)
    g = build_from_spec(spec, t)
    xd = to_dev(t["x"], "f16")
    x64 = to_f64(t["x"], "f16")
    w64 = to_f64(t["w"][0], "f16")
    b64 = t["b"][0].astype(np.float64)
    rng = np.random.default_rng(si)
    idx = np.stack([rng.integers(0, 32, 3000), rng.integers(0, c, 3000),
                    rng.integers(0, hw, 3000), rng.integers(0, hw, 3000)], axis=1)
    ref = O.round_to(O.conv2d_points(x64, w64, b64, idx, 1, 1, 1, "none"), "f16")
    import torch
    for rt in g.routines(1):
        g.set_path([0, rt["id"]])
        y = g.run(xd)
        torch.cuda.synchronize()
        y = from_dev(y, "f16")
        got = y[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]]
        e = err(got, ref, "f16")
        print(f"sweep c{c} {rt['name']} err {e:.2e}", flush=True)
        assert e <= TOL["f16"], rt["name"]
    g.close()


def test_hip_graph_replays_match_eager():
    import torch
    spec = resnet18(1)
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.select("fixed", "NHWC", "igemm")
    eager, xd = run_out(g, spec, t)
    g.set_option(N.OPT_HIPGRAPH, 1)
    for rep in range(4):
        y = g.run(xd)
        torch.cuda.synchronize()
        got = from_dev(y, "bf16").reshape(1, -1)
        assert np.array_equal(got, eager), rep
        junk = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
    g.close()
