"""Selection oracle: the optimal routine path by exhaustive enumeration.

TEST INFRASTRUCTURE ONLY.  It restates Definitions 1 and 2 of the paper
(Sec. IV-A): a routine path picks one routine per layer and, on every edge
whose endpoint routines have different schemas, the adapt routine of that
edge; its time is the sum of the times of its members, and the optimal path
minimises it.  Layer 0 is the auxiliary input layer and the last layer the
auxiliary output layer (Sec. IV-E), each with one zero-time routine.

Readings taken where the paper is silent:
* one adapt per edge (Definition 1 charges each edge separately);
* an adapt between equal schemas costs 0 (the void adapt of Sec. IV-F);
* ties are broken by the tuple of routine ids in layer order, so the optimum
  is unique: the key is (T, tuple).

A problem is a dict::

    {"n_layers": L,
     "routines": [[(rid, schema, ns), ...] for each layer 0..L-1],   # ns None = unavailable
     "edges": [(j, i, A), ...]}   # A[a][b] = adapt time schema a -> b, None = unavailable

``exhaustive`` enumerates every routine combination.  ``blockwise`` is an
independent exact solver for nets that decompose into a chain of blocks
between cut layers (layers every input-to-output path passes); it enumerates
the schemas of each block's interior exhaustively and chains the blocks.
"""

from __future__ import annotations

import itertools
import json


def path_time(problem, choice):
    """T(S) of a full routine choice (tuple of indices into each layer's list)."""
    rts = problem["routines"]
    total = 0
    for i, ci in enumerate(choice):
        ns = rts[i][ci][2]
        if ns is None:
            return None
        total += ns
    for j, i, A in problem["edges"]:
        a = rts[j][choice[j]][1]
        b = rts[i][choice[i]][1]
        if a == b:
            continue
        c = A[a][b]
        if c is None:
            return None
        total += c
    return total


def exhaustive(problem):
    """Returns (T, tuple of routine ids, number of paths enumerated)."""
    rts = problem["routines"]
    best = None
    count = 0
    for choice in itertools.product(*[range(len(r)) for r in rts]):
        count += 1
        t = path_time(problem, choice)
        if t is None:
            continue
        key = (t, tuple(rts[i][c][0] for i, c in enumerate(choice)))
        if best is None or key < best:
            best = key
    if best is None:
        return None, None, count
    return best[0], best[1], count


def _fastest_in_schema(routines, schema):
    """F_i(lambda) of Eq. (1): the fastest routine of the schema, lowest id on ties."""
    best = None
    for rid, sc, ns in routines:
        if sc != schema or ns is None:
            continue
        if best is None or (ns, rid) < best:
            best = (ns, rid)
    return best


def cut_layers(problem):
    """Layers that no edge jumps over (every input-output path passes them)."""
    n = problem["n_layers"]
    jumped = [False] * n
    for j, i, _ in problem["edges"]:
        for v in range(j + 1, i):
            jumped[v] = True
    return [v for v in range(n) if not jumped[v]]


def blockwise(problem, schemas):
    """Exact optimum for nets whose layers are numbered so that every block
    between consecutive cut layers is a contiguous id range.  Returns (T, tuple)."""
    n = problem["n_layers"]
    rts = problem["routines"]
    cuts = cut_layers(problem)
    assert cuts[0] == 0 and cuts[-1] == n - 1
    F = [{s: _fastest_in_schema(rts[i], s) for s in schemas} for i in range(n)]
    edges_by_to = {}
    for j, i, A in problem["edges"]:
        edges_by_to.setdefault(i, []).append((j, A))

    def edge_cost(assign, i):
        tot = 0
        for j, A in edges_by_to.get(i, []):
            a, b = assign[j], assign[i]
            if a == b:
                continue
            if A[a][b] is None:
                return None
            tot += A[a][b]
        return tot

    # state: schema of the current cut -> (T, tuple of routine ids so far, schema assignment)
    state = {}
    for s in schemas:
        f = F[0][s]
        if f is not None:
            state[s] = (f[0], (f[1],), {0: s})
    for u, v in zip(cuts[:-1], cuts[1:]):
        interior = list(range(u + 1, v))
        new = {}
        for su, (tu, tup, asg) in state.items():
            for combo in itertools.product(schemas, repeat=len(interior) + 1):
                a = dict(asg)
                t = tu
                ids = []
                ok = True
                for layer, sc in zip(interior + [v], combo):
                    f = F[layer][sc]
                    if f is None:
                        ok = False
                        break
                    a[layer] = sc
                    t += f[0]
                    ids.append(f[1])
                    ec = edge_cost(a, layer)
                    if ec is None:
                        ok = False
                        break
                    t += ec
                if not ok:
                    continue
                key = (t, tup + tuple(ids))
                sv = combo[-1]
                if sv not in new or key < new[sv][:2]:
                    new[sv] = (key[0], key[1], {v: sv})
        state = new
    best = min((val[0], val[1]) for val in state.values())
    return best


def problem_from_costs(costs):
    """Build a problem from the cost-table JSON the library exports (a dict or a
    JSON string): layers with their routines and times, edges with their
    adapt-time matrices (-1 = unavailable).  A routine's schema is its layout
    when the matrices are 3 x 3 (one element type), else its (dtype, layout)
    schema index, which the 9 x 9 matrices are indexed by."""
    if isinstance(costs, str):
        costs = json.loads(costs)
    layers = sorted(costs["layers"], key=lambda d: d["id"])
    by_schema = any(len(e["ns"]) == 9 for e in costs["edges"])
    routines = []
    for d in layers:
        rl = []
        for r in d["routines"]:
            ns = r["ns"]
            rl.append((r["rid"], r["schema"] if by_schema else r["layout"], None if ns < 0 else ns))
        routines.append(rl)
    edges = []
    for e in costs["edges"]:
        A = [[None if v < 0 else v for v in row] for row in e["ns"]]
        edges.append((e["from"], e["to"], A))
    return {"n_layers": len(routines), "routines": routines, "edges": edges}


def childnet_time(rows):
    """Time and sub-routine choice of a routine built from sub-layers (a
    childnet, Sec. III-D): ``rows[s]`` lists the times of sub-layer s's
    sub-routines (None or a negative value = unavailable).  The sub-layers
    form a chain passing tensors of one fixed format (no adapts), so a
    choice's time is the sum of its members' times; every choice is
    enumerated and the minimum (ties: the lowest tuple of indices) returned,
    or (None, None) when some sub-layer has no available sub-routine."""
    best = None
    for choice in itertools.product(*[range(len(r)) for r in rows]):
        ts = [rows[s][q] for s, q in enumerate(choice)]
        if any(t is None or t < 0 for t in ts):
            continue
        key = (sum(ts), choice)
        if best is None or key < best:
            best = key
    return (None, None) if best is None else best
