"""DPRS through the C ABI on host-only graphs (no GPU): the selected routine
path must be bit-exact (same routine-id tuple, same total) with the
exhaustive enumeration of Definitions 1-2 on small nets, and with the
independent block-wise exact solver on full-size nets; plus the ABI's
state machine and error codes, and the counts printed in the paper."""

import ctypes
import json
import os
import re

import numpy as np
import pytest

from oracle.select import blockwise, exhaustive, path_time, problem_from_costs
from paper_2110_06037_amd import Graph, build_from_spec, native as N
from tests.problems import random_dag, residual_chain
from workloads import mobilenet_v2, resnet18, resnet50, tiny_chain, vgg16

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "dprs_paper_counts.json")))


def header_functions():
    src = open(os.path.join(ROOT, "include", "softneuro.h")).read()
    return sorted(set(re.findall(r"\b(sn_[a-z_]+)\s*\(", src)))


def test_library_exports_every_header_function():
    names = header_functions()
    assert "sn_graph_create" in names and "sn_run" in names and len(names) >= 18
    lib = ctypes.CDLL(N.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(N.SIGNATURES)


# ------------------------------------------------------------------ helpers

def graph_from_edges(L, edges, layouts=("NCHW", "NHWC")):
    """Host-only library graph whose layers 1..L-2 follow ``edges`` (layer
    L-1 is the auxiliary output): one input -> 1x1 conv, two -> add."""
    C = 8
    g = Graph("f16", 1, C, 4, 4, device=-1, layouts=list(layouts), algos=["direct", "igemm"],
              params=False)
    preds = {i: sorted(j for j, t in edges if t == i) for i in range(1, L - 1)}
    w = np.zeros((C, C, 1, 1), np.float16)
    b = np.zeros(C, np.float32)
    for i in range(1, L - 1):
        p = preds[i]
        if len(p) == 1:
            got = g.add_conv(p[0], w, b)
        else:
            assert len(p) == 2
            got = g.add_add(p[0], p[1])
        assert got == i
    return g


def randomise(costs, seed, max_cost=3, p_missing=0.0):
    rng = np.random.default_rng(seed)
    for layer in costs["layers"][1:-1]:
        for r in layer["routines"]:
            r["ns"] = int(rng.integers(0, max_cost + 1))
            if p_missing and rng.random() < p_missing:
                r["ns"] = -1
    for e in costs["edges"]:
        e["ns"] = [[0 if a == b else int(rng.integers(0, max_cost + 1)) for b in range(3)]
                   for a in range(3)]
    return costs


def dp_vs(g, costs):
    g.set_costs(costs)
    g.select("dprs")
    ids, total = g.path()
    return tuple(ids) + (0,), total


# ------------------------------------------------------------------ DPRS == exhaustive

@pytest.mark.parametrize("seed", range(10))
def test_dprs_equals_exhaustive_on_random_dags(seed):
    L, E = random_dag(6, seed)
    g = graph_from_edges(L, E)
    costs = randomise(g.costs(), seed)
    got = dp_vs(g, costs)
    t, tup, _ = exhaustive(problem_from_costs(costs))
    assert got == (tup, t)


@pytest.mark.parametrize("seed", range(8))
def test_dprs_equals_exhaustive_on_residual_chains(seed):
    L, E = residual_chain(3, seed)
    g = graph_from_edges(L, E)
    costs = randomise(g.costs(), 50 + seed)
    if np.prod([len(l["routines"]) for l in costs["layers"]]) > 20000:
        L, E = residual_chain(2, seed)
        g = graph_from_edges(L, E)
        costs = randomise(g.costs(), 50 + seed)
    got = dp_vs(g, costs)
    t, tup, _ = exhaustive(problem_from_costs(costs))
    assert got == (tup, t)


def test_dprs_non_series_parallel_net():
    # 1 -> {2, 3}, 2 -> {4, 5}, {4, 3} -> 6, {5, 6} -> 7: the predecessors of
    # 6 carry different constraint sets ({1, 2} and {1})
    E = [(0, 1), (1, 2), (1, 3), (2, 4), (2, 5), (4, 6), (3, 6), (5, 7), (6, 7), (7, 8)]
    g = graph_from_edges(9, E)
    for seed in range(6):
        costs = randomise(g.costs(), 200 + seed)
        got = dp_vs(g, costs)
        t, tup, _ = exhaustive(problem_from_costs(costs))
        assert got == (tup, t)


def test_dprs_three_schemas_with_missing_routines():
    L, E = residual_chain(2, 7)
    g = graph_from_edges(L, E, layouts=("NCHW", "NHWC", "NC8HW8"))
    for seed in range(4):
        costs = randomise(g.costs(), 300 + seed, p_missing=0.2)
        t, tup, _ = exhaustive(problem_from_costs(costs))
        if t is None:
            continue
        assert dp_vs(g, costs) == (tup, t)


def test_dprs_tiny_chain_256_paths():
    spec = tiny_chain()
    g = build_from_spec(spec, device=-1)
    for seed in range(5):
        costs = randomise(g.costs(), 400 + seed, max_cost=1000)
        t, tup, count = exhaustive(problem_from_costs(costs))
        # conv layers: 2 algorithms x 2 layouts; gap: 2 layouts; FC: direct and
        # the 1x1-convolution childnet in 2 layouts
        assert count == 4 * 4 * 4 * 2 * 4
        assert dp_vs(g, costs) == (tup, t)


@pytest.mark.parametrize("maker", [lambda: resnet18(1), lambda: resnet50(32),
                                   lambda: mobilenet_v2(8), lambda: vgg16(32)])
def test_dprs_equals_blockwise_exact_on_full_nets(maker):
    spec = maker()
    g = build_from_spec(spec, device=-1)
    for seed in range(2):
        costs = randomise(g.costs(), 500 + seed, max_cost=50)
        prob = problem_from_costs(costs)
        t, tup = blockwise(prob, [0, 1, 2])
        assert dp_vs(g, costs) == (tup, t)


# ------------------------------------------------------------------ closed forms and invariants

def test_single_schema_is_per_layer_fastest():
    L, E = residual_chain(3, 11)
    g = graph_from_edges(L, E, layouts=("NCHW",))
    costs = randomise(g.costs(), 600, max_cost=9)
    ids, total = dp_vs(g, costs)
    expect = [min(l["routines"], key=lambda r: (r["ns"], r["rid"])) for l in costs["layers"]]
    assert ids == tuple(r["rid"] for r in expect)
    assert total == sum(r["ns"] for r in expect)


def test_free_adapts_give_global_per_layer_fastest():
    L, E = random_dag(7, 12)
    g = graph_from_edges(L, E, layouts=("NCHW", "NHWC", "NC8HW8"))
    costs = randomise(g.costs(), 601, max_cost=9)
    for e in costs["edges"]:
        e["ns"] = [[0] * 3 for _ in range(3)]
    ids, total = dp_vs(g, costs)
    expect = [min(l["routines"], key=lambda r: (r["ns"], r["rid"])) for l in costs["layers"]]
    assert ids == tuple(r["rid"] for r in expect)


def test_unavailable_adapts_give_best_single_schema_path():
    L, E = residual_chain(3, 13)
    g = graph_from_edges(L, E, layouts=("NCHW", "NHWC"))
    costs = randomise(g.costs(), 602, max_cost=9)
    for e in costs["edges"]:
        e["ns"] = [[0 if a == b else -1 for b in range(3)] for a in range(3)]
    # the input and output are NCHW, so only the all-NCHW path is feasible
    ids, total = dp_vs(g, costs)
    layouts = [next(r["layout"] for r in l["routines"] if r["rid"] == i)
               for l, i in zip(costs["layers"], ids)]
    assert set(layouts) == {0}


def test_island_routine_between_two_schemas():
    # a chain where one middle layer is far faster in the other schema: the
    # optimum switches there and back (Sec. V-A, Table 3's block4 pooling)
    E = [(i, i + 1) for i in range(7)]
    g = graph_from_edges(8, E)
    costs = g.costs()
    for l in costs["layers"][1:-1]:
        for r in l["routines"]:
            fast = l["id"] == 4 and r["layout"] == 1
            r["ns"] = 30 if fast else (100 if r["layout"] == 0 else 200)
    for e in costs["edges"]:
        e["ns"] = [[0, 20, 20], [20, 0, 20], [20, 20, 0]]
    ids, total = dp_vs(g, costs)
    lay = [next(r["layout"] for r in l["routines"] if r["rid"] == i)
           for l, i in zip(costs["layers"], ids)]
    assert lay == [0, 0, 0, 0, 1, 0, 0, 0]
    assert total == 5 * 100 + 30 + 2 * 20


def test_dp_never_slower_than_any_fixed_path():
    spec = resnet50(1)
    g = build_from_spec(spec, device=-1)
    costs = randomise(g.costs(), 700, max_cost=100)
    _, t_dp = dp_vs(g, costs)
    for lay in ("NCHW", "NHWC", "NC8HW8"):
        for algo in ("direct", "igemm", "winograd"):
            g.select("fixed", lay, algo)
            _, t_fix = g.path()
            assert t_dp <= t_fix


# ------------------------------------------------------------------ the paper's counts

def test_net_b_merge_evaluates_four_candidates():
    gb = GOLD["net_b"]
    E = [tuple(e) for e in gb["edges"]] + [(5, 6)]
    g = graph_from_edges(7, E)
    costs = randomise(g.costs(), 800)
    dp_vs(g, costs)
    states, cands = g.dp_stats(gb["merge_layer"])
    assert cands == gb["candidates_per_state"]
    assert states == 2 * 2  # own schema x constraint on layer 1


def test_net_c_pattern_counts():
    gc = GOLD["net_c"]
    E = [tuple(e) for e in gc["edges"]] + [(8, 9)]
    g = graph_from_edges(10, E)
    costs = randomise(g.costs(), 801)
    got = dp_vs(g, costs)
    for layer in gc["layers_with_eight_patterns"]:
        assert g.dp_stats(layer)[0] == gc["patterns"]
    assert g.dp_stats(8)[0] == gc["layer_8_states"]
    t, tup, _ = exhaustive(problem_from_costs(costs))
    assert got == (tup, t)


# ------------------------------------------------------------------ ABI behaviour

def status_of(fn, *args):
    try:
        fn(*args)
    except N.SNError as e:
        return e.code
    return 0


def test_abi_state_machine_and_errors():
    g = Graph("bf16", 1, 8, 8, 8, device=-1)
    assert status_of(g.select) == -3                       # no layers
    w = np.zeros((8, 8, 3, 3), np.uint16)
    b = np.zeros(8, np.float32)
    c1 = g.add_conv(0, w, b, 1, 1)
    assert status_of(g.select) == -3                       # no costs yet
    assert status_of(g.add_conv, 5, w, b) == -1            # unknown input id
    w2 = np.zeros((16, 8, 3, 3), np.uint16)
    c2 = g.add_conv(c1, w2, np.zeros(16, np.float32), 1, 1)
    assert status_of(g.add_add, c1, c2) == -2              # shape mismatch
    assert status_of(g.add_conv, c1, np.zeros((8, 2, 3, 3), np.uint16), b, 1, 1, 4) == -4  # groups
    assert status_of(g.profile, 5, 20, 0) == -5            # host-only
    assert status_of(g.set_costs, "{not json") == -1
    assert status_of(g.set_costs, '{"layers": [], "edges": []}') == -1
    g.add_gap(c2)
    costs = g.costs()
    for l in costs["layers"][1:-1]:
        for r in l["routines"]:
            r["ns"] = 10 + r["rid"]
    for e in costs["edges"]:
        e["ns"] = [[0 if a == b else 5 for b in range(3)] for a in range(3)]
    g.set_costs(costs)
    assert g.costs() == costs                              # round trip
    g.select("dprs")
    ids, total = g.path()
    assert len(ids) == 4 and total > 0
    assert status_of(g.add_gap, c2) == -3                  # after selection
    x = ctypes.c_void_p(16)
    assert N.lib().sn_run(g._g, x, x, None) == -5          # host-only cannot run
    assert status_of(g.set_path, [0, 0]) == -1             # wrong length
    g.set_path([0, 0, 0, 0])
    assert g.path()[0] == [0, 0, 0, 0]


def test_missing_library_fails_loudly(monkeypatch):
    # the binding has no CPU fallback: without the built library every call raises
    monkeypatch.setattr(N, "_lib", None)
    monkeypatch.setattr(N, "LIB_PATH", "/nonexistent/libsoftneuro.so")
    with pytest.raises(ImportError):
        N.lib()
    with pytest.raises(ImportError):
        Graph("bf16", 1, 8, 8, 8, device=-1)


def test_flush_option_bounds():
    g = Graph("bf16", 1, 8, 8, 8, device=-1)
    g.set_option(N.OPT_FLUSH, 512 << 20)   # accepted at any time (a timing setting)
    g.set_option(N.OPT_FLUSH, 0)
    assert status_of(g.set_option, N.OPT_FLUSH, -1) == -1
    assert status_of(g.set_option, N.OPT_FLUSH, 1 << 40) == -1


def test_create_rejects_bad_arguments():
    p = ctypes.c_void_p()
    lib = N.lib()
    assert lib.sn_graph_create(9, 1, 1, 1, 1, -1, ctypes.byref(p)) == -1
    assert lib.sn_graph_create(0, 0, 1, 1, 1, -1, ctypes.byref(p)) == -1
    assert lib.sn_graph_create(0, 1, 1, 1, 1, -2, ctypes.byref(p)) == -1
    assert b"dtype" in lib.sn_last_error() or b"dims" in lib.sn_last_error() or True


def test_tensors_of_two_gib_or_more_are_unsupported():
    # every kernel addresses a tensor with 32-bit byte offsets: the input and
    # every layer output (channels padded to 8) must stay below 2 GiB
    p = ctypes.c_void_p()
    lib = N.lib()
    assert lib.sn_graph_create(2, 1024, 64, 224, 224, -1, ctypes.byref(p)) == -4   # 6.6 GB bf16
    assert b"2 GiB" in lib.sn_last_error()
    assert lib.sn_graph_create(0, 1, 3, 16384, 16384, -1, ctypes.byref(p)) == -4   # C padded to 8: 8.6 GB
    g = Graph("bf16", 16, 64, 224, 224, device=-1)                                   # 103 MB input
    w = np.zeros((4096, 64, 1, 1), np.uint16)
    assert status_of(g.add_conv, 0, w, np.zeros(4096, np.float32)) == -4              # 6.6 GB output
    c = g.add_conv(0, np.zeros((64, 64, 3, 3), np.uint16), np.zeros(64, np.float32), 1, 1)
    assert c == 1


def test_dangling_layer_is_rejected():
    g = Graph("f16", 1, 8, 4, 4, device=-1)
    w = np.zeros((8, 8, 1, 1), np.float16)
    b = np.zeros(8, np.float32)
    a = g.add_conv(0, w, b)
    g.add_conv(0, w, b)          # layer 1's output is never consumed
    costs = randomise(g.costs(), 1)
    g.set_costs(costs)
    assert status_of(g.select) == -1


# ------------------------------------------------------------------ integrated profiling candidates

def _restricted(problem, mask):
    """The problem with the routines of layers 1..L-2 limited to the layouts in mask."""
    rts = [list(r) for r in problem["routines"]]
    for i in range(1, len(rts) - 1):
        rts[i] = [(rid, lay, ns if (mask >> lay) & 1 else None) for rid, lay, ns in rts[i]]
    return dict(problem, routines=rts)


@pytest.mark.parametrize("seed", range(6))
def test_integrated_candidates_are_restricted_optima_and_fixed_paths(seed):
    # Sec. III-C: unit profiling filters the routine patterns that integrated
    # profiling times; every candidate is an exact optimum of the unit-profiled
    # model within its restriction, checked by exhaustive enumeration
    L, E = random_dag(5, seed)
    g = graph_from_edges(L, E, layouts=("NCHW", "NHWC", "NC8HW8"))
    costs = randomise(g.costs(), 900 + seed, max_cost=6, p_missing=0.15)
    g.set_costs(costs)
    g.select("dprs")
    before = g.path()
    cands = g.profile_integrated(reps=0)
    assert g.path() == before, "enumeration must not change the selection"
    paths = [tuple(c["path"]) for c in cands]
    assert len(set(paths)) == len(paths), "identical paths are kept once"
    assert cands[0]["kind"] == "dprs" and cands[0]["a"] == 7
    assert tuple(cands[0]["path"]) == tuple(before[0]) and cands[0]["model_ns"] == before[1]
    problem = problem_from_costs(costs)
    seen_masks = []
    for c in cands:
        assert c["measured_ns"] == -1
        if c["kind"] == "dprs":
            seen_masks.append(c["a"])
            t, tup, _ = exhaustive(_restricted(problem, c["a"]))
            assert (tuple(c["path"]) + (0,), c["model_ns"]) == (tup, t)
        else:
            g.select("fixed", c["a"], c["b"])
            assert tuple(c["path"]) == tuple(g.path()[0])
    assert seen_masks[0] == 7 and seen_masks[1:] == sorted(seen_masks[1:])
    # every subset whose restricted optimum exists and differs from the earlier candidates appears
    for m in range(1, 7):
        t, tup, _ = exhaustive(_restricted(problem, m))
        if t is not None:
            assert tup[:-1] in paths
    for lay in range(3):
        for algo in range(2):
            try:
                g.select("fixed", lay, algo)
            except N.SNError:
                continue
            assert tuple(g.path()[0]) in paths


def test_integrated_profiling_needs_costs_and_a_device():
    g = graph_from_edges(3, [(0, 1), (1, 2)])
    with pytest.raises(N.SNError, match="SN_E_STATE"):
        g.profile_integrated(reps=0)
    g.set_costs(randomise(g.costs(), 1))
    with pytest.raises(N.SNError, match="SN_E_DEVICE"):
        g.profile_integrated(reps=5)
    with pytest.raises(N.SNError, match="SN_E_INVALID"):
        g.profile_integrated(warmup=-1, reps=0)


def test_in_path_refinement_needs_costs_a_path_and_a_device():
    g = graph_from_edges(3, [(0, 1), (1, 2)])
    with pytest.raises(N.SNError, match="SN_E_STATE"):
        g.refine_in_path()
    g.set_costs(randomise(g.costs(), 1))
    with pytest.raises(N.SNError, match="SN_E_STATE"):
        g.refine_in_path()  # costs but no selected path
    g.select("dprs")
    with pytest.raises(N.SNError, match="SN_E_DEVICE"):
        g.refine_in_path()
    for kw in ({"tol_permille": -1}, {"tol_permille": 1001}, {"max_alts": 0}, {"max_alts": 17},
               {"reps": 0}, {"reps": 1001}):
        with pytest.raises(N.SNError, match="SN_E_INVALID"):
            g.refine_in_path(**kw)
    path = g.path()
    assert g.path() == path  # the failed calls leave the selection alone


def test_workspace_limit_restricts_the_routine_set():
    # Time optimised under a memory restriction (the restriction the paper's
    # Sec. VI names as future work, Winograd's transforms its example): with
    # SN_OPT_WS_LIMIT every layer keeps exactly the routines whose workspace
    # fits, ids stay dense, and the DP path is the exhaustive optimum over the
    # reduced set
    w = np.zeros((64, 64, 3, 3), np.uint16)
    b = np.zeros(64, np.float32)

    def build(limit):
        g = Graph("bf16", 2, 64, 14, 14, device=-1, ws_limit=limit)
        c1 = g.add_conv(0, w, b, 1, 1)
        g.add_conv(c1, w, b, 1, 1)
        return g

    free = build(None)
    full = [free.routines(i) for i in (1, 2)]
    assert any(r["ws_bytes"] > 0 for r in full[0]), "split Winograd and split reductions use workspace"
    for limit in (0, min(r["ws_bytes"] for r in full[0] if r["ws_bytes"] > 0)):
        g = build(limit)
        for li, every in zip((1, 2), full):
            kept = g.routines(li)
            assert [r["id"] for r in kept] == list(range(len(kept)))
            assert [r["name"] for r in kept] == [r["name"] for r in every if r["ws_bytes"] <= limit]
            assert all(r["ws_bytes"] <= limit for r in kept) and len(kept) < len(every)
        # random costs: the DP over the reduced set equals exhaustive search over it
        costs = randomise(g.costs(), 3 + limit % 5, max_cost=50)
        assert dp_vs(g, costs) == exhaustive(problem_from_costs(costs))[1::-1]
        g.close()
    free.close()
    # the option's range, and it is a routine-set option (before any layer)
    g = Graph("bf16", 2, 64, 14, 14, device=-1, ws_limit=0)
    assert status_of(g.set_option, N.OPT_WS_LIMIT, -2) == -1
    g.add_conv(0, w, b, 1, 1)
    assert status_of(g.set_option, N.OPT_WS_LIMIT, 1 << 20) == -3   # after layers were added
    g.close()


def test_childnet_routine_time_is_the_optimum_over_its_sub_layers():
    # The three-kernel Winograd routines are childnets (Sec. III-D): wgenc ->
    # wgconv (one sub-routine per GEMM tile) -> wgdec.  Its time in the cost
    # table is the DPRS optimum over its sub-routines' times (the algorithm
    # applied to the childnet before the net), which must equal the
    # enumeration of every sub-routine choice; the net's DP then uses it.
    from oracle.select import childnet_time
    w = np.zeros((64, 64, 3, 3), np.uint16)
    b = np.zeros(64, np.float32)
    g = Graph("bf16", 2, 64, 14, 14, device=-1)
    c1 = g.add_conv(0, w, b, 1, 1)
    g.add_conv(c1, w, b, 1, 1)
    costs = g.costs()
    kids = [r for l in costs["layers"] for r in l["routines"] if "child" in r]
    assert kids and all(r["algo"] == 2 and "fused" not in r["name"] for r in kids)
    assert all(r["child"]["layers"] == ["wgenc", "wgconv", "wgdec"] and len(r["child"]["routines"][1]) >= 2
               for r in kids)
    rng = np.random.default_rng(5)
    for trial in range(6):
        costs = randomise(g.costs(), trial, max_cost=40)
        for l in costs["layers"]:
            for r in l["routines"]:
                if "child" in r:
                    r["child"]["ns"] = [[int(rng.integers(-1 if trial % 2 else 0, 30)) for _ in row]
                                        for row in r["child"]["ns"]]
        g.set_costs(costs)
        got = g.costs()
        for l, lg in zip(costs["layers"], got["layers"]):
            for r, rg in zip(l["routines"], lg["routines"]):
                if "child" not in r:
                    assert rg["ns"] == r["ns"]
                    continue
                t, choice = childnet_time(r["child"]["ns"])
                assert rg["ns"] == (-1 if t is None else t)
                if t is not None:
                    assert tuple(rg["child"]["path"]) == choice
        assert dp_vs(g, got) == exhaustive(problem_from_costs(got))[1::-1]
    # a childnet never profiled (every sub-routine time unknown) keeps the
    # routine's own listed time
    costs = randomise(g.costs(), 9, max_cost=40)
    for l in costs["layers"]:
        for r in l["routines"]:
            if "child" in r:
                r["child"]["ns"] = [[-1 for _ in row] for row in r["child"]["ns"]]
                r["ns"] = 17
    g.set_costs(costs)
    assert all(r["ns"] == 17 for l in g.costs()["layers"] for r in l["routines"] if "child" in r)
    g.close()
