"""Random routine-selection problems (graphs + integer cost tables) for the tests.

Only structure and seeded integers live here; no selection arithmetic.
"""

import numpy as np

SCHEMAS3 = [0, 1, 2]


def random_dag(n_mid, seed, max_preds=2):
    """A 1-in-1-out DAG with layers 0..n_mid+1 (0 = input, last = output)."""
    g = np.random.default_rng(seed)
    L = n_mid + 2
    edges = set()
    for i in range(1, L - 1):
        k = int(g.integers(1, max_preds + 1))
        preds = g.choice(i, size=min(k, i), replace=False)
        for j in preds:
            edges.add((int(j), i))
    # every middle layer must reach the output
    has_succ = {j for j, _ in edges}
    for j in range(1, L - 1):
        if j not in has_succ:
            # connect to a random later middle layer or the output
            i = int(g.integers(j + 1, L))
            edges.add((j, i))
    if not any(i == L - 1 for _, i in edges):
        edges.add((L - 2, L - 1))
    # the output takes exactly one input: funnel everything into the last middle layer
    outs = [j for j, i in edges if i == L - 1]
    if len(outs) > 1:
        edges = {(j, i) for (j, i) in edges if i != L - 1}
        last = L - 2
        for j in outs:
            if j != last:
                edges.add((j, last))
        edges.add((last, L - 1))
    return L, sorted(edges)


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
