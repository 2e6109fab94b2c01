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
from workloads import (CONV_SWEEP_SHAPES, conv_sweep, decode, fuse_projection, fuse_residual, generate, mobilenet_v2,
                       resnet18, resnet50, tiny_chain, to_f64, vgg16, with_batch)

pytestmark = pytest.mark.gpu


def decoded(t, dtype):
    return decode(t, dtype)


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
    # cache-cold unit profiling (median of single runs after a flush): a
    # complete positive cost table, cached apart from the warm one (so a warm
    # profile afterwards gives back the warm table), and its DP path is again
    # the exhaustive optimum of that table and matches the oracle
    g.set_option(N.OPT_FLUSH, 64 << 20)
    g.profile(warmup=1, reps=5)
    g.set_option(N.OPT_FLUSH, 0)
    cold = g.costs()
    for l in cold["layers"][1:-1]:
        assert all(r["ns"] > 0 for r in l["routines"]), l
    g.select("dprs")
    ids, total = g.path()
    tt, tup, _ = exhaustive(problem_from_costs(cold))
    assert tuple(ids) + (0,) == tup and total == tt
    out, _ = run_out(g, spec, t)
    assert err(out, ref, "f32") <= TOL["f32"]
    g.profile(warmup=3, reps=10)
    assert g.costs() == costs


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


def test_in_path_refinement_keeps_schemas_and_parity():
    # in-path refinement swaps a layer's routine only for one of the same
    # schema whose unit-profiled time is within the tolerance of the selected
    # one's, so the adapts stay as they were and the output still matches the
    # oracle
    spec = fuse_projection(fuse_residual(resnet50(2, "bf16")))
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    before, _ = g.path()
    n = g.refine_in_path(tol_permille=200, max_alts=3, reps=5)
    after, total = g.path()
    changed = [i for i in range(len(after)) if after[i] != before[i]]
    print("refined layers", changed, [g.routines(i)[after[i]]["name"] for i in changed], flush=True)
    assert n == len(changed)
    for i in changed:
        r0, r1 = g.routines(i)[before[i]], g.routines(i)[after[i]]
        assert r1["schema"] == r0["schema"]
        assert r1["cost_ns"] <= r0["cost_ns"] * 1.2 + 1
    out, _ = run_out(g, spec, t)
    assert err(out, oracle_out(spec, t), spec["dtype"]) <= TOL[spec["dtype"]]
    g.close()


@pytest.mark.parametrize("name", ["resnet18", "mobilenetv2", "resnet50_bf16", "resnet50_f16",
                                  "resnet50_fused", "resnet50_proj", "mobilenetv2_fused", "vgg16_64px"])
def test_net_dp_and_fixed_paths_match_oracle(name):
    spec = {"resnet18": lambda: resnet18(1), "mobilenetv2": lambda: mobilenet_v2(1),
            "vgg16_64px": lambda: vgg16(2, "bf16", 64),
            "resnet50_bf16": lambda: resnet50(1, "bf16"),
            "resnet50_f16": lambda: resnet50(1, "f16"),
            "resnet50_fused": lambda: fuse_residual(resnet50(1, "bf16")),
            "resnet50_proj": lambda: fuse_projection(fuse_residual(resnet50(1, "bf16"))),
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


def test_workspace_limited_selection_runs_within_the_limit():
    # memory-restricted tuning: with no routine workspace allowed, the
    # profiled DP path of a bs2 ResNet-18 (split-reduction tiles and the
    # three-kernel Winograd left out) uses none, and matches the oracle
    spec = fuse_projection(fuse_residual(resnet18(2, "bf16")))
    t = generate(spec)
    free = build_from_spec(spec, t)
    g = build_from_spec(spec, t, ws_limit=0)
    n_layers = len(spec["layers"]) + 1
    assert sum(len(g.routines(i)) for i in range(1, n_layers)) < sum(len(free.routines(i)) for i in range(1, n_layers))
    free.close()
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    ids, _ = g.path()
    assert all(g.routines(i)[ids[i]]["ws_bytes"] == 0 for i in range(1, n_layers))
    out, _ = run_out(g, spec, t)
    e = err(out, oracle_out(spec, t), "bf16")
    print(f"resnet18 bs2 workspace-free dprs err {e:.3e}", flush=True)
    assert e <= TOL["bf16"]
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


def _images_out(g, spec, t, images):
    import torch
    xd = to_dev(t["x"], spec["dtype"])
    y = g.run(xd)
    torch.cuda.synchronize()
    out = from_dev(y, spec["dtype"]).reshape(spec["batch"], -1)
    d = decoded(t, spec["dtype"])
    d["x"] = d["x"][images]
    ref = O.forward(with_batch(spec, len(images)), d, storage="dtype")[-1]
    return out, out[images], ref.reshape(len(images), -1)


FULL_BATCH = {
    # name: (spec factory, images through the oracle: first, middle, last)
    "resnet50_bs32_bf16_proj": (lambda: fuse_projection(fuse_residual(resnet50(32, "bf16"))), [0, 13, 31]),
    "resnet50_bs32_f16_proj": (lambda: fuse_projection(fuse_residual(resnet50(32, "f16"))), [1, 19, 30]),
    "resnet50_bs32_bf16_fused": (lambda: fuse_residual(resnet50(32, "bf16")), [0, 13, 31]),
    "resnet50_bs32_f16_fused": (lambda: fuse_residual(resnet50(32, "f16")), [0, 17, 31]),
    "resnet50_bs32_f16": (lambda: resnet50(32, "f16"), [2, 31]),
    "mobilenetv2_bs8_fused": (lambda: fuse_residual(mobilenet_v2(8)), [0, 3, 7]),
    "mobilenetv2_bs8": (lambda: mobilenet_v2(8), [1, 6]),
    "vgg16_bs32_224": (lambda: vgg16(32, "bf16"), [0, 31]),
}


@pytest.mark.parametrize("name", list(FULL_BATCH))
def test_full_batch_paths_on_images_across_the_batch(name):
    # the benchmark's configurations at their full batch: the DPRS path and
    # the path integrated profiling keeps (the one bench.py times), checked
    # on images at the start, middle and end of the batch, so that tiles far
    # from the first of every persistent workgroup are compared too
    make, images = FULL_BATCH[name]
    spec = make()
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.profile(warmup=2, reps=5)
    g.select("dprs")
    out, got, ref = _images_out(g, spec, t, images)
    e = err(got, ref, spec["dtype"])
    print(f"{name} dprs images {images} err {e:.3e}", flush=True)
    assert e <= TOL[spec["dtype"]]
    assert np.all(np.isfinite(out))
    dprs_ids = g.path()[0]
    g.profile_integrated(warmup=2, reps=3)
    if g.path()[0] != dprs_ids:
        out, got, ref2 = _images_out(g, spec, t, images)
        e = err(got, ref, spec["dtype"])
        print(f"{name} selected path images {images} err {e:.3e}", flush=True)
        assert e <= TOL[spec["dtype"]]
        assert np.all(np.isfinite(out))
    g.close()


def _rotating_layout_path(g):
    # a routine of layout (i mod 3) on layer i where one exists (implicit
    # GEMM first): a converter on almost every edge
    ids = [0]
    for i in range(1, g.num_layers()):
        rts = g.routines(i)
        want = [r for r in rts if r["layout"] == i % 3] or rts
        ids.append(min(want, key=lambda r: (r["algo"] != 1, r["id"]))["id"])
    return ids


def test_run_timed_equals_run_on_a_mixed_layout_path():
    # sn_run_timed repeats every layer's converters and routine; a converter's
    # source must outlive the layer's routine, so the repeated run gives the
    # same bits as sn_run on a path that switches layout on every edge
    import torch
    spec = resnet18(1)
    t = generate(spec)
    g = build_from_spec(spec, t)
    ids = _rotating_layout_path(g)
    g.set_path(ids)
    layouts = [g.routines(i)[ids[i]]["layout"] for i in range(len(ids))]
    assert len(set(layouts[1:])) == 3
    out, xd = run_out(g, spec, t)
    assert err(out, oracle_out(spec, t), "bf16") <= TOL["bf16"]
    for reps in (3, 1):
        y, ms = g.run_timed(xd, reps=reps)
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(y, "bf16").reshape(1, -1), out), reps
        assert all(m > 0 for m in ms[1:])
    g.close()


def odd_channel_net():
    """Channel counts that are not multiples of 8 on every layer: NC8HW8
    stores them padded."""
    L = [
        {"type": "conv", "in": [0], "k": 12, "r": 3, "s": 3, "stride": 1, "pad": 1, "groups": 1, "act": "relu"},
        {"type": "conv", "in": [1], "k": 12, "r": 3, "s": 3, "stride": 2, "pad": 1, "groups": 12, "act": "relu6"},
        {"type": "conv", "in": [2], "k": 20, "r": 1, "s": 1, "stride": 1, "pad": 0, "groups": 1, "act": "none"},
        {"type": "maxpool", "in": [3], "k": 3, "stride": 1, "pad": 1},
        {"type": "conv", "in": [4], "k": 20, "r": 3, "s": 3, "stride": 1, "pad": 1, "groups": 1, "act": "none"},
        {"type": "add", "in": [5, 3], "act": "relu"},
        # a 1x1 convolution with a folded residual input (layer 4)
        {"type": "conv", "in": [6, 4], "k": 20, "r": 1, "s": 1, "stride": 1, "pad": 0, "groups": 1, "act": "relu"},
        {"type": "gap", "in": [7]},
        {"type": "fc", "in": [8], "k": 10},
    ]
    return {"name": "odd_channels", "dtype": "bf16", "batch": 3, "in_chw": [3, 13, 11],
            "input_dist": "uniform", "seed": 5, "layers": L,
            "layouts": ["NCHW", "NHWC", "NC8HW8"], "algos": ["direct", "igemm", "winograd"]}


@pytest.mark.parametrize("algo", ["igemm", "direct", "winograd"])
def test_nc8hw8_stored_outputs_keep_padded_channels_zero(algo):
    # every layer's output as its NC8HW8 routine stored it: the channels
    # padded up to a multiple of 8 hold exact zeros, and the real channels
    # hold the oracle's layer output
    import torch
    spec = odd_channel_net()
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.set_option(N.OPT_KEEP, 1)
    g.select("fixed", "NC8HW8", algo)
    xd = to_dev(t["x"], "bf16")
    y = g.run(xd)
    torch.cuda.synchronize()
    refs = O.forward(spec, decoded(t, "bf16"), storage="dtype", keep=True)
    for i in range(1, g.num_layers()):
        n, c, h, w = g.layer_shape(i)
        try:
            buf, lay = g.layer_output(i)
        except N.SNError as e:
            assert i == g.num_layers() - 1 and e.code == -4, e   # stored into the user's output
            continue
        torch.cuda.synchronize()
        assert lay == N.NC8HW8
        c8 = (c + 7) // 8 * 8
        bits = buf.cpu().numpy().view(np.uint16)
        assert bits.size == n * c8 * h * w, (i, bits.size)
        blk = bits.reshape(n, c8 // 8, h, w, 8).transpose(0, 1, 4, 2, 3).reshape(n, c8, h, w)
        assert not np.any(blk[:, c:]), f"layer {i}: padded channels hold non-zero bits"
        got = to_f64(blk[:, :c], "bf16")
        e = err(got, refs[i].reshape(n, c, h, w), "bf16")
        print(f"odd-channel net {algo} layer {i} err {e:.2e}", flush=True)
        assert e <= TOL["bf16"], i
    out = from_dev(y, "bf16").reshape(3, -1)
    assert err(out, refs[-1].reshape(3, -1), "bf16") <= TOL["bf16"]
    g.close()


def test_plan_launch_list_matches_the_routines():
    # sn_plan_launches lists a run's kernel launches by layer without
    # launching anything: every layer appears in order, a Winograd layer
    # with its three kernels (input transform, tile GEMMs, output transform),
    # converters before the layer they feed; the next run is unaffected
    import torch
    spec = resnet18(1)
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.select("fixed", "NHWC", "winograd")
    out0, xd = run_out(g, spec, t)
    ids = g.path()[0]
    lay = g.plan_launches()
    assert lay == sorted(lay) and set(lay) == set(range(1, g.num_layers()))
    for i in range(1, g.num_layers()):
        rt = g.routines(i)[ids[i]]
        n = lay.count(i)
        conv = 1 if i == 1 else 0          # the input's NCHW -> NHWC converter feeds layer 1
        if rt["algo"] == N.WINOGRAD:
            assert n == 3 + conv, (i, rt["name"], n)
        elif i == 1:
            assert n == 2, (i, rt["name"], n)
    out1, _ = run_out(g, spec, t)
    assert np.array_equal(out0, out1)
    g.close()
