"""Random routine-selection problems (graphs + integer cost tables) for the tests.

Only structure and seeded integers live here; no selection arithmetic.
"""

import numpy as np

SCHEMAS3 = [0, 1, 2]


def random_dag(n_mid, seed, max_preds=2):
    """A 1-in-1-out DAG with layers 0..n_mid+1 (0 = input, last = output):
    every middle layer has 1..max_preds inputs and at least one consumer,
    and the output takes the last middle layer.  Rejection-sampled."""
    L = n_mid + 2
    for attempt in range(1000):
        g = np.random.default_rng(seed * 1000 + attempt)
        edges = set()
        indeg = [0] * L
        for i in range(1, L - 1):
            k = int(g.integers(1, max_preds + 1))
            for j in g.choice(i, size=min(k, i), replace=False):
                edges.add((int(j), i))
                indeg[i] += 1
        edges.add((L - 2, L - 1))
        indeg[L - 1] = 1
        ok = True
        for j in range(0, L - 2):
            if any(a == j for a, _ in edges):
                continue
            later = [i for i in range(j + 1, L - 1) if indeg[i] < max_preds]
            if not later:
                ok = False
                break
            i = int(g.choice(later))
            edges.add((j, i))
            indeg[i] += 1
        if ok:
            return L, sorted(edges)
    raise RuntimeError("no DAG found")


def residual_chain(n_blocks, seed):
    """Series-parallel net: a chain of plain layers and residual blocks
    (identity or projection shortcut), numbered in insertion order."""
    g = np.random.default_rng(seed)
    edges = []
    cur = 0
    nxt = 1
    for _ in range(n_blocks):
        kind = int(g.integers(0, 3))
        if kind == 0:                      # plain layer
            edges.append((cur, nxt))
            cur, nxt = nxt, nxt + 1
        else:
            a, b = nxt, nxt + 1
            edges += [(cur, a), (a, b)]
            nxt += 2
            sc = cur
            if kind == 2:                  # projection shortcut
                sc = nxt
                edges.append((cur, sc))
                nxt += 1
            m = nxt
            edges += [(b, m), (sc, m)]
            cur, nxt = m, nxt + 1
    out = nxt
    edges.append((cur, out))
    return out + 1, edges


def random_costs(L, edges, seed, schemas=SCHEMAS3, max_routines=2, max_cost=3,
                 fixed_io=True):
    """Routine lists and adapt matrices with small integer costs (forces ties)."""
    g = np.random.default_rng(seed)
    S = len(schemas)
    routines = []
    for i in range(L):
        if fixed_io and (i == 0 or i == L - 1):
            routines.append([(0, 0, 0)])
            continue
        rl = []
        rid = 0
        for s in schemas:
            for _ in range(int(g.integers(1, max_routines + 1))):
                rl.append((rid, s, int(g.integers(0, max_cost + 1))))
                rid += 1
        routines.append(rl)
    E = []
    for j, i in edges:
        A = [[0 if a == b else int(g.integers(0, max_cost + 1)) for b in range(S)] for a in range(S)]
        E.append((j, i, A))
    return {"n_layers": L, "routines": routines, "edges": E}
