"""Precision-hybrid schemas and multi-input/multi-output nets on host-only
graphs (no GPU).

Hybrid tuning (Sec. IV-F) makes a schema a (dtype, layout) pair: with
float32, float16 and bfloat16 allowed a layer has up to 9 schemas, and
adapts cast between element types as well as converting layouts.  DPRS is
unchanged, so its path must stay bit-exact with the exhaustive enumeration
of Definitions 1-2 on the same cost table.  Multi-input/multi-output nets
are joined by zero-cost auxiliary input and output layers (Sec. IV-E); the
DP must again equal the exhaustive optimum."""

import json

import numpy as np
import pytest

from oracle.select import exhaustive, path_time, problem_from_costs
from paper_2110_06037_amd import Graph, build_from_spec, native as N
from tests.problems import random_dag, residual_chain
from workloads import net_d, resnet18, tiny_chain

ALL3 = ["f32", "f16", "bf16"]


def hybrid_graph(L, edges, dtypes, layouts=("NCHW", "NHWC", "NC8HW8"), io="f16"):
    """Host-only graph of 1x1 convolutions (one input) and adds (two inputs)
    following ``edges``, with one routine per schema (implicit GEMM, one
    parameter) and the given element types allowed."""
    C = 8
    g = Graph(io, 1, C, 4, 4, device=-1, layouts=list(layouts), algos=["igemm"], params=False,
              dtypes=dtypes)
    preds = {i: sorted(j for j, t in edges if t == i) for i in range(1, L - 1)}
    w = np.zeros((C, C, 1, 1), {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}[io])
    b = np.zeros(C, np.float32)
    for i in range(1, L - 1):
        p = preds[i]
        got = g.add_conv(p[0], w, b) if len(p) == 1 else g.add_add(p[0], p[1])
        assert got == i
    return g


def randomise_schemas(costs, seed, max_cost=4):
    """Small random integer times (forcing ties) for every routine and for
    every adapt between two schemas that some routine uses."""
    rng = np.random.default_rng(seed)
    used = set()
    for layer in costs["layers"]:
        for r in layer["routines"]:
            used.add(r["schema"] if len(costs["edges"][0]["ns"]) == 9 else r["layout"])
        if layer["type"] in (N.L_INPUT, N.L_OUTPUT):
            continue
        for r in layer["routines"]:
            r["ns"] = int(rng.integers(0, max_cost + 1))
    for e in costs["edges"]:
        S = len(e["ns"])
        e["ns"] = [[0 if a == b else (int(rng.integers(0, max_cost + 1)) if a in used and b in used else -1)
                    for b in range(S)] for a in range(S)]
    return costs


def dp(g, costs):
    g.set_costs(costs)
    g.select("dprs")
    ids, total = g.path()
    return tuple(ids) + (0,), total


def test_routines_per_dtype_and_schema_fields():
    g = hybrid_graph(3, [(0, 1), (1, 2)], ALL3, io="bf16")
    rts = g.routines(1)
    assert len(rts) == 9
    # the run dtype first, then the others in sn_dtype order; layouts within
    assert [(r["dtype"], r["layout"]) for r in rts] == [(2, 0), (2, 1), (2, 2), (0, 0), (0, 1), (0, 2),
                                                        (1, 0), (1, 1), (1, 2)]
    assert all(r["schema"] == 3 * r["dtype"] + r["layout"] for r in rts)
    assert rts[0]["name"].startswith("bf16:") and rts[3]["name"].startswith("f32:")
    costs = g.costs()
    assert all(len(e["ns"]) == 9 for e in costs["edges"])
    # a single-dtype graph keeps its layout-indexed 3 x 3 table and plain names
    g1 = hybrid_graph(3, [(0, 1), (1, 2)], None, io="bf16")
    c1 = g1.costs()
    assert all(len(e["ns"]) == 3 for e in c1["edges"])
    assert [r["name"] for r in g1.routines(1)] == ["nchw/igemm:p0", "nhwc/igemm:p0", "nc8hw8/igemm:p0"]


@pytest.mark.parametrize("dtypes,layouts", [(["f16", "bf16"], ("NCHW", "NHWC", "NC8HW8")),
                                            (ALL3, ("NCHW", "NHWC")),
                                            (ALL3, ("NCHW", "NHWC", "NC8HW8"))])
@pytest.mark.parametrize("seed", range(4))
def test_hybrid_dprs_equals_exhaustive(dtypes, layouts, seed):
    # |Lambda| = 6, 6 and 9 schemas
    n_mid = 3 if len(dtypes) * len(layouts) == 9 else 4
    L, E = random_dag(n_mid, 40 + seed)
    g = hybrid_graph(L, E, dtypes, layouts)
    costs = randomise_schemas(g.costs(), 7 * seed + len(dtypes))
    t, tup, count = exhaustive(problem_from_costs(costs))
    assert count == (len(dtypes) * len(layouts)) ** n_mid
    assert dp(g, costs) == (tup, t)


@pytest.mark.parametrize("seed", range(3))
def test_hybrid_dprs_on_a_residual_chain(seed):
    L, E = residual_chain(2, seed)
    g = hybrid_graph(L, E, ["f32", "bf16"], ("NHWC", "NC8HW8"))
    costs = randomise_schemas(g.costs(), 90 + seed)
    t, tup, _ = exhaustive(problem_from_costs(costs))
    assert dp(g, costs) == (tup, t)


def test_hybrid_special_cases():
    L, E = random_dag(4, 3)
    g = hybrid_graph(L, E, ALL3, ("NCHW", "NHWC"))
    costs = g.costs()
    # casts free -> every layer takes its own fastest routine
    costs = randomise_schemas(costs, 5)
    for e in costs["edges"]:
        e["ns"] = [[0 if v >= 0 else -1 for v in row] for row in e["ns"]]
    ids, total = dp(g, costs)
    best = [min(l["routines"], key=lambda r: (r["ns"], r["rid"])) for l in costs["layers"]]
    assert total == sum(r["ns"] for r in best)
    # casts forbidden -> one dtype on every layer: the run dtype's NCHW at the
    # ends pins it to the run dtype
    costs = randomise_schemas(g.costs(), 6)
    for e in costs["edges"]:
        e["ns"] = [[0 if a == b else (v if a // 3 == b // 3 and v >= 0 else -1) for b, v in enumerate(row)]
                   for a, row in enumerate(e["ns"])]
    ids, total = dp(g, costs)
    assert {g.routines(i)[ids[i]]["dtype"] for i in range(len(ids) - 1)} == {N.F16}


def test_hybrid_cost_table_round_trip_and_fixed_paths():
    g = hybrid_graph(5, [(0, 1), (1, 2), (2, 3), (3, 4)], ["f32", "bf16"], ("NCHW", "NHWC"), io="bf16")
    costs = randomise_schemas(g.costs(), 11)
    g.set_costs(json.dumps(costs))
    assert g.costs() == costs
    g.select("fixed", "NHWC", "igemm")
    ids, _ = g.path()
    assert all(g.routines(i)[ids[i]]["dtype"] == N.BF16 and g.routines(i)[ids[i]]["layout"] == N.NHWC
               for i in range(1, len(ids)))
    # integrated profiling lists the per-dtype DPRS paths among its
    # candidates: float32 is fast on odd layers, bfloat16 on even ones, so
    # the hybrid optimum mixes them and differs from both one-dtype optima
    for l in costs["layers"][1:-1]:
        for r in l["routines"]:
            r["ns"] = 1 if (r["dtype"] == N.F32) == (l["id"] % 2 == 1) else 9
    for e in costs["edges"]:
        e["ns"] = [[v if v < 0 or a == b else (1 if a % 3 == b % 3 else 3) for b, v in enumerate(row)]
                   for a, row in enumerate(e["ns"])]
    g.set_costs(costs)
    g.select("dprs")
    hybrid_dtypes = [g.routines(i)[g.path()[0][i]]["dtype"] for i in (1, 2, 3)]
    assert hybrid_dtypes == [N.F32, N.BF16, N.F32]
    cands = g.profile_integrated(reps=0)
    masks = [(c["a"], c["b"]) for c in cands if c["kind"] == "dprs"]
    assert masks[0] == (3, 5) and (3, 1) in masks and (3, 4) in masks
    bad = dict(costs)
    bad["edges"] = [dict(e, ns=[[0, 1, 2], [1, 0, 2], [2, 2, 0]]) for e in costs["edges"]]
    with pytest.raises(N.SNError):
        g.set_costs(bad)


def test_dtypes_option_rules():
    g = Graph("bf16", 1, 8, 4, 4, device=-1)
    with pytest.raises(N.SNError):
        g.set_option(N.OPT_DTYPES, 0)
    with pytest.raises(N.SNError):
        g.set_option(N.OPT_DTYPES, 8)
    g.set_option(N.OPT_DTYPES, 1)        # float32 routines only, bf16 tensors at the ends
    g.add_conv(0, np.zeros((8, 8, 1, 1), np.uint16), np.zeros(8, np.float32))
    assert {r["dtype"] for r in g.routines(1)} == {N.F32}
    with pytest.raises(N.SNError):
        g.set_option(N.OPT_DTYPES, 7)     # routine-set options only before layers
    costs = randomise_schemas(g.costs(), 1)
    g.set_costs(costs)
    g.select("dprs")
    g.select("fixed", "NCHW", "igemm")    # the lowest allowed dtype
    assert g.routines(1)[g.path()[0][1]]["dtype"] == N.F32


# ------------------------------------------------------------------ multi-input / multi-output

def test_net_d_structure():
    spec = net_d()
    g = build_from_spec(spec, device=-1)
    assert g.num_io() == (2, 2)
    costs = g.costs()
    edges = [(e["from"], e["to"]) for e in costs["edges"]]
    aux_out = g.num_layers()
    assert (0, 2) in edges                                   # auxiliary input -> second input
    assert (7, aux_out) in edges and (8, aux_out) in edges   # both outputs -> auxiliary output
    assert [r["name"] for r in g.routines(2)] == ["input/nchw"]
    # the structural edge carries no cost
    e02 = next(e for e in costs["edges"] if (e["from"], e["to"]) == (0, 2))
    assert e02["ns"][0][0] == 0


@pytest.mark.parametrize("seed", range(5))
def test_net_d_dprs_equals_exhaustive(seed):
    spec = net_d()
    g = build_from_spec(spec, device=-1, layouts=["NCHW", "NHWC"], algos=["igemm"], params=False)
    costs = randomise_schemas(g.costs(), 300 + seed)
    t, tup, _ = exhaustive(problem_from_costs(costs))
    assert dp(g, costs) == (tup, t)
    assert path_time(problem_from_costs(costs), tuple(
        next(k for k, r in enumerate(l["routines"]) if r["rid"] == rid)
        for l, rid in zip(sorted(costs["layers"], key=lambda d: d["id"]), tup))) == t


def test_mimo_with_hybrid_dtypes_equals_exhaustive():
    spec = net_d()
    g = build_from_spec(spec, device=-1, layouts=["NHWC"], algos=["igemm"], params=False,
                        dtypes=["f16", "bf16"])
    for seed in range(3):
        costs = randomise_schemas(g.costs(), 500 + seed)
        t, tup, _ = exhaustive(problem_from_costs(costs))
        assert dp(g, costs) == (tup, t)


def test_mimo_rules():
    g = Graph("f16", 2, 3, 8, 8, device=-1)
    x1 = g.add_input(4, 8, 8)
    w = np.zeros((4, 3, 1, 1), np.float16)
    a = g.add_conv(0, w, np.zeros(4, np.float32))
    m = g.add_add(a, x1)
    with pytest.raises(N.SNError):
        g.mark_output(x1)                 # an input cannot be an output
    g.mark_output(m)
    with pytest.raises(N.SNError):
        g.mark_output(m)                  # marked twice
    b = g.add_conv(m, np.zeros((4, 4, 1, 1), np.float16), np.zeros(4, np.float32))
    # b reaches no output: selection refuses the net
    costs = randomise_schemas(g.costs(), 1)
    g.set_costs(costs)
    with pytest.raises(N.SNError) as e:
        g.select("dprs")
    assert e.value.code == -1 and "output" in str(e.value)
    g2 = Graph("f16", 1, 3, 8, 8, device=-1)
    with pytest.raises(N.SNError):
        g2.add_input(0, 8, 8)
