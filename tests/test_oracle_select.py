"""Pins of the selection oracle (exhaustive enumeration of Definitions 1-2).

Checked against closed forms the paper states or implies: with one schema the
optimum is each layer's fastest routine (Sec. IV, opening paragraph); with
free adaptation it is each layer's global fastest; with impossible adaptation
it is the best single-schema path; a cheap isolated schema switch (the
``block4 pooling`` situation of Sec. V-A, Table 3) is taken when it pays; and
the independent block-wise exact solver agrees with enumeration.
"""

import itertools

import numpy as np
import pytest

from oracle.select import blockwise, cut_layers, exhaustive, path_time
from tests.problems import random_costs, random_dag, residual_chain


def chain_edges(L):
    return [(i, i + 1) for i in range(L - 1)]


def test_enumeration_count_is_product_of_routine_counts():
    p = random_costs(6, chain_edges(6), seed=1)
    _, _, count = exhaustive(p)
    assert count == int(np.prod([len(r) for r in p["routines"]]))


def test_single_schema_is_per_layer_argmin():
    g = np.random.default_rng(2)
    L = 7
    routines = [[(0, 0, 0)]] + [[(r, 0, int(g.integers(0, 9))) for r in range(4)]
                                for _ in range(L - 2)] + [[(0, 0, 0)]]
    p = {"n_layers": L, "routines": routines,
         "edges": [(j, i, [[0]]) for j, i in chain_edges(L)]}
    t, tup, _ = exhaustive(p)
    expect = [min(rl, key=lambda r: (r[2], r[0])) for rl in routines]
    assert tup == tuple(r[0] for r in expect)
    assert t == sum(r[2] for r in expect)


def test_free_adapts_give_global_per_layer_argmin():
    L, E = random_dag(5, seed=3)
    p = random_costs(L, E, seed=4, max_routines=1)
    for e in p["edges"]:
        for row in e[2]:
            row[:] = [0] * len(row)
    t, tup, _ = exhaustive(p)
    expect = [min(rl, key=lambda r: (r[2], r[0])) for rl in p["routines"]]
    assert tup == tuple(r[0] for r in expect)
    assert t == sum(r[2] for r in expect)


def test_forbidden_adapts_give_best_single_schema_path():
    L, E = residual_chain(2, seed=5)
    p = random_costs(L, E, seed=6, fixed_io=False, max_routines=1)
    for e in p["edges"]:
        A = e[2]
        for a in range(3):
            for b in range(3):
                A[a][b] = 0 if a == b else None
    t, tup, _ = exhaustive(p)
    best = None
    for s in range(3):
        tot, ids = 0, []
        for rl in p["routines"]:
            cand = [r for r in rl if r[1] == s]
            r = min(cand, key=lambda r: (r[2], r[0]))
            tot += r[2]
            ids.append(r[0])
        key = (tot, tuple(ids))
        best = key if best is None or key < best else best
    assert (t, tup) == best


def test_island_switch_is_selected():
    # chain of 5 middle layers; schema 1 is much faster on layer 3 only and
    # switching there and back costs less than it saves
    L = 7
    routines = [[(0, 0, 0)]]
    for i in range(1, 6):
        routines.append([(0, 0, 10), (1, 1, 3 if i == 3 else 20)])
    routines.append([(0, 0, 0)])
    A = [[0, 2], [2, 0]]
    p = {"n_layers": L, "routines": routines, "edges": [(j, i, A) for j, i in chain_edges(L)]}
    t, tup, _ = exhaustive(p)
    assert tup == (0, 0, 0, 1, 0, 0, 0)
    assert t == 4 * 10 + 3 + 2 + 2
    # a switch-once heuristic (one schema change at most) cannot produce it
    assert sum(1 for a, b in zip(tup[1:], tup[2:]) if a != b) == 2


def test_net_b_hand_worked():
    # Net B of Sec. IV-C: 1 branches to 3 (via 2) and 4, merging at 5.
    # layers: 0 in, 1, 2, 3, 4, 5, 6 out ; edges 0-1, 1-2, 2-3, 1-4, 3-5, 4-5, 5-6
    E = [(0, 1), (1, 2), (2, 3), (1, 4), (3, 5), (4, 5), (5, 6)]
    c = {1: (5, 6), 2: (5, 1), 3: (5, 1), 4: (1, 5), 5: (5, 5)}
    routines = [[(0, 0, 0)]] + [[(0, 0, c[i][0]), (1, 1, c[i][1])] for i in range(1, 6)] + [[(0, 0, 0)]]
    A = [[0, 1], [1, 0]]
    p = {"n_layers": 7, "routines": routines, "edges": [(j, i, A) for j, i in E]}
    t, tup, _ = exhaustive(p)
    # by hand: layers 2, 3 want schema b (cost 1 each), layer 4 wants schema a.
    # 1:a, 2:b, 3:b, 4:a, 5:a -> 5 + 1 + 1 + 1 + 5 = 13 plus adapts 1->2 and
    # 3->5 (1 each) = 15.  Alternatives: 5:b costs 13 + adapts 1->2, 4->5, 5->6
    # = 16; 1:b costs 14 + adapts 0->1, 1->4, 3->5 = 17; all-a costs 21.
    assert t == 15
    assert tup == (0, 0, 1, 1, 0, 0, 0)


@pytest.mark.parametrize("seed", range(12))
def test_blockwise_equals_exhaustive_on_residual_chains(seed):
    L, E = residual_chain(3, seed)
    p = random_costs(L, E, seed=100 + seed, max_routines=1)
    t, tup, _ = exhaustive(p)
    assert blockwise(p, [0, 1, 2]) == (t, tup)


def test_cut_layers_of_residual_block():
    # 0 -> 1 -> 2 -> 4, 0 -> 3 -> 4 (projection), 4 -> 5
    p = {"n_layers": 6, "routines": [[(0, 0, 0)]] * 6,
         "edges": [(0, 1, None), (1, 2, None), (2, 4, None), (0, 3, None), (3, 4, None),
                   (4, 5, None)]}
    assert cut_layers(p) == [0, 4, 5]


def test_path_time_counts_each_edge_once():
    routines = [[(0, 0, 0)], [(0, 1, 2)], [(0, 1, 3)], [(0, 0, 0)]]
    A = [[0, 7], [5, 0]]
    p = {"n_layers": 4, "routines": routines,
         "edges": [(0, 1, A), (0, 2, A), (1, 3, A), (2, 3, A)]}
    # two edges 0->{1,2} adapt 0->1 (7 each), two edges {1,2}->3 adapt 1->0 (5 each)
    assert path_time(p, (0, 0, 0, 0)) == 2 + 3 + 7 + 7 + 5 + 5


def test_childnet_time_hand_worked():
    # a chain of sub-layers with one format between them: the time of a
    # choice is the sum of its sub-routines' times, the minimum over choices
    # (ties to the lowest index tuple), unavailable when a sub-layer has none
    from oracle.select import childnet_time
    assert childnet_time([[3], [5, 2, 7], [4]]) == (9, (0, 1, 0))
    assert childnet_time([[3, 1], [5, None, 2], [4]]) == (7, (1, 2, 0))
    assert childnet_time([[1], [2, 2], [0]]) == (3, (0, 0, 0))          # tie: lowest tuple
    assert childnet_time([[1], [-1, None], [0]]) == (None, None)        # wgconv unavailable
    assert childnet_time([[0]]) == (0, (0,))
