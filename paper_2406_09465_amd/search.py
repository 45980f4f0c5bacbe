"""Plan construction over the candidate kernels of Algorithm 1.

``random_plan`` draws a valid ordered plan from the supported candidates (the
kernels whose profiling cost is finite): it repeatedly picks a candidate whose
inputs are all available and that materializes something new, until every
graph output exists.  Plans built this way may execute primitives redundantly
and skip dead ones, as the orchestration problem allows (Section 4.2).
"""

from __future__ import annotations

import random


class GraphView:
    """Python-side structure of a finalized graph (ops, operands, consumers)."""

    def __init__(self, graph):
        self.g = graph
        n = graph.num_nodes()
        self.op = {}
        self.ins = {}
        for i in range(n):
            self.op[i] = graph.node_info(i)[0]
            self.ins[i] = graph.node_inputs(i)
        self.cons = {i: [] for i in range(n)}
        for v in range(n):
            for u in self.ins[v]:
                self.cons[u].append(v)
        self.inputs = [i for i in range(n) if self.op[i] == "input"]
        self.outputs = graph.outputs()

    def external(self, prims):
        s = set(prims)
        return {u for v in prims for u in self.ins[v] if u not in s}


def random_plan(view: GraphView, cands, rng: random.Random, max_kernels=64):
    avail = set(view.inputs)

    def is_avail(u):
        if u in avail:
            return True
        return view.op[u] == "reshape" and is_avail(view.ins[u][0])

    ext = [view.external(p) for p, _ in cands]
    plan = []
    for _ in range(max_kernels):
        if all(is_avail(o) for o in view.outputs):
            return plan
        ready = [i for i, (p, o) in enumerate(cands)
                 if all(is_avail(u) for u in ext[i]) and any(not is_avail(x) for x in o)]
        if not ready:
            raise RuntimeError("no candidate can make progress")
        i = rng.choice(ready)
        plan.append((list(cands[i][0]), list(cands[i][1])))
        avail |= set(cands[i][1])
    raise RuntimeError("plan did not cover the graph outputs")


def sampled_plans(graph, n, seed, max_prims=12, max_outs=2):
    """``n`` seeded random valid plans built from supported candidates."""
    cands = graph.candidates(max_prims=max_prims, max_outs=max_outs, only_supported=True)
    view = GraphView(graph)
    rng = random.Random(seed)
    return [random_plan(view, cands, rng) for _ in range(n)]
