"""Kernel-orchestration definitions as plain set computations (Korch, Section 4).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Only primitives are nodes of the primitive graph here; graph inputs are
tensors that every kernel may read.  All functions work on an oracle
``Graph`` and sets of node indices.
"""

from __future__ import annotations

from itertools import combinations


def prim_edges(g):
    """Edges (p1, p2) between primitives (graph-input nodes are excluded)."""
    prims = set(g.primitives())
    return [(u, v) for (u, v) in g.edges() if u in prims and v in prims]


def reach(g):
    """reach[u] = set of primitives reachable from u by a non-empty path."""
    prims = g.primitives()
    succ = {p: set() for p in prims}
    for u, v in prim_edges(g):
        succ[u].add(v)
    out = {}
    for p in reversed(prims):  # creation order is topological
        r = set()
        for s in succ[p]:
            r.add(s)
            r |= out[s]
        out[p] = r
    return out


def is_convex(g, nodes, _reach=None):
    """Definition 1: no p1, p2 in P' and q outside P' with p1 ~> q ~> p2."""
    nodes = set(nodes)
    r = _reach or reach(g)
    for q in g.primitives():
        if q in nodes:
            continue
        if any(q in r[p1] for p1 in nodes) and any(p2 in r[q] for p2 in nodes):
            return False
    return True


def is_execution_state(g, nodes):
    """Definition 2: closed under predecessors (every edge into the set starts in it)."""
    nodes = set(nodes)
    return all(u in nodes for (u, v) in prim_edges(g) if v in nodes)


def execution_states_bruteforce(g):
    """Every predecessor-closed subset, by enumerating all subsets (tiny graphs only)."""
    prims = g.primitives()
    out = set()
    for k in range(len(prims) + 1):
        for c in combinations(prims, k):
            if is_execution_state(g, c):
                out.add(frozenset(c))
    return out


def execution_states_search(g):
    """The state search of Algorithm 1: grow states one ready primitive at a time.

    Starting from the empty state, a primitive whose predecessors are all in
    the current state may be added; every state reached is recorded once.
    (An explicit work list replaces the recursion; the set reached is the same.)
    """
    prims = g.primitives()
    preds = {p: set() for p in prims}
    for u, v in prim_edges(g):
        preds[v].add(u)
    seen = {frozenset()}
    stack = [frozenset()]
    while stack:
        x = stack.pop()
        for v in prims:
            if v not in x and preds[v] <= x:
                x2 = x | {v}
                if x2 not in seen:
                    seen.add(x2)
                    stack.append(x2)
    return seen


def theorem1_witness(g, nodes):
    """The two execution states constructed in the proof of Theorem 1.

    P1 = P' closed under predecessors; P2 = S closed under predecessors, where
    S are the outside primitives with an edge into P'.  For convex P',
    P' = P1 minus P2.
    """
    nodes = set(nodes)
    preds = {p: set() for p in g.primitives()}
    for u, v in prim_edges(g):
        preds[v].add(u)

    def closure(seed):
        out = set(seed)
        work = list(seed)
        while work:
            x = work.pop()
            for u in preds[x]:
                if u not in out:
                    out.add(u)
                    work.append(u)
        return out

    s = {u for (u, v) in prim_edges(g) if v in nodes and u not in nodes}
    return closure(nodes), closure(s)


def convex_sets_from_states(states):
    """Every non-empty difference D2 minus D1 of states with D1 a proper subset of D2."""
    out = set()
    for d1 in states:
        for d2 in states:
            if d1 < d2:
                out.add(frozenset(d2 - d1))
    return out


def is_possible_output_set(g, kernel, outs):
    """Definition 3, with graph outputs counted as read outside every kernel.

    Every u in O has an edge (u, v) with v outside P', or u is a graph output.
    """
    kernel = set(kernel)
    cons = g.consumers()
    gouts = set(g.outputs)
    for u in outs:
        if u not in kernel:
            return False
        if u in gouts:
            continue
        if not any(v not in kernel for v in cons[u]):
            return False
    return True


def external_inputs(g, kernel):
    """Tensors a kernel reads: producers u outside P' of edges (u, v) with v in P'."""
    kernel = set(kernel)
    return {u for v in kernel for u in g.nodes[v].inputs if u not in kernel}


def plan_is_valid(g, plan):
    """Validity of an ordered plan (list of ``(prims, outs)``).

    Checks, per kernel: non-empty convex primitive set, a non-empty possible
    output set (Definition 3); the dependency constraint with ordering (every
    external primitive read is materialized by an EARLIER kernel, or is a
    reshape of something available); and the output constraint (every graph
    output is materialized by some kernel, or is a reshape of an available
    tensor).  Returns ``(ok, reason)``.
    """
    r = reach(g)
    prims = set(g.primitives())
    avail = {i for i, n in enumerate(g.nodes) if n.op == "input"}

    def is_avail(u):
        if u in avail:
            return True
        n = g.nodes[u]
        return n.op == "reshape" and is_avail(n.inputs[0])

    for k, (kp, ko) in enumerate(plan):
        kp = set(kp)
        if not kp or not kp <= prims:
            return False, f"kernel {k}: empty or contains a non-primitive"
        if not is_convex(g, kp, r):
            return False, f"kernel {k}: not convex"
        if not ko or not is_possible_output_set(g, kp, ko):
            return False, f"kernel {k}: bad output set"
        for u in external_inputs(g, kp):
            if not is_avail(u):
                return False, f"kernel {k}: input {g.nodes[u].name} not produced earlier"
        avail |= set(ko)
    for o in g.outputs:
        if not is_avail(o):
            return False, f"graph output {g.nodes[o].name} not produced"
    return True, ""
