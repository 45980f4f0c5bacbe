"""Measured-cost kernel orchestration (Korch, Section 4.2 with Algorithm 1).

Candidates are the kernels (P', O) that Algorithm 1 enumerates and a kernel
family implements; the cost of a candidate is its latency measured in isolation
by the profiler (a candidate no family implements has infinite cost and is
dropped).  The chooser returns the cheapest *ordered* plan: a sequence of
candidates in which every kernel's external inputs are graph inputs or outputs
of earlier kernels (a reshape of an available tensor is available as a view),
and after which every graph output is available.

Each such sequence satisfies the output and dependency constraints of the binary
program of Section 4.2, and conversely every feasible kernel set that admits an
execution order is such a sequence, with the same total cost.  The optimum is
found exactly as a shortest path over "availability states" (the set of tensors
materialized so far) with Dijkstra's algorithm.  A primitive may be computed by
several kernels (redundant execution) and primitives no output needs are never
computed (pruning), as the program allows.
"""

from __future__ import annotations

import heapq
import time
from dataclasses import dataclass, field

from .search import GraphView


@dataclass
class Choice:
    kernels: list                 # [(prims, outs)] in execution order
    cost_us: float                # sum of the chosen kernels' measured latencies
    states: int                   # availability states expanded by the search
    candidates: int               # candidates with a finite cost
    costs: dict = field(default_factory=dict)   # (prims, outs) -> us
    failures: list = field(default_factory=list)  # candidates whose kernel did not compile


def _masks(view: GraphView):
    views = sorted((v, view.ins[v][0]) for v in view.op if view.op[v] == "reshape")

    def closure(m: int) -> int:
        for v, src in views:  # node ids are topological: one pass suffices
            if m >> src & 1:
                m |= 1 << v
        return m

    start = 0
    for v in view.inputs:
        start |= 1 << v
    goal = 0
    for v in view.outputs:
        goal |= 1 << v
    return closure, closure(start), goal


def choose(view: GraphView, cands, costs) -> Choice:
    """Cheapest ordered plan.  ``cands``: [(prims, outs)]; ``costs``: [us or None]."""
    closure, start, goal = _masks(view)
    usable = []
    for (p, o), c in zip(cands, costs):
        if c is None:
            continue
        ext = 0
        for u in view.external(p):
            ext |= 1 << u
        out = 0
        for v in o:
            out |= 1 << v
        usable.append((ext, out, float(c), (tuple(p), tuple(o))))
    dist = {start: 0.0}
    parent = {start: None}
    heap = [(0.0, 0, start)]
    tie = 1
    expanded = 0
    while heap:
        d, _, m = heapq.heappop(heap)
        if d > dist[m]:
            continue
        expanded += 1
        if m & goal == goal:
            seq = []
            while parent[m] is not None:
                m, k = parent[m]
                seq.append(k)
            seq.reverse()
            return Choice(kernels=[(list(p), list(o)) for p, o in seq], cost_us=d, states=expanded,
                          candidates=len(usable))
        for ext, out, c, key in usable:
            if ext & ~m or not out & ~m:
                continue
            m2 = closure(m | out)
            d2 = d + c
            if d2 < dist.get(m2, float("inf")):
                dist[m2] = d2
                parent[m2] = (m, key)
                heapq.heappush(heap, (d2, tie, m2))
                tie += 1
    raise RuntimeError("no ordered plan of the candidates covers the graph outputs")


def plan_cost(view: GraphView, kernels, cost_of) -> float:
    """Total measured cost of a given plan (each kernel looked up in ``cost_of``)."""
    return sum(cost_of[(tuple(p), tuple(o))] for p, o in kernels)


def profile_candidates(graph, cands, warmup=10, reps=100, flush_bytes=512 << 20, log=None, failures=None, db=None):
    """Measured latency (us) of every candidate on the current device, None when
    no family implements it.  A candidate whose generated kernel fails to
    compile also costs infinity; it is appended to ``failures`` when given.
    With a ``ProfileDB`` (``db``), candidates measured before under the same
    protocol on the same kind of device are looked up instead of profiled, and
    new measurements are recorded."""
    from ._abi import E_COMPILE, KorchError
    costs = []
    t0 = time.time()
    dev = None
    if db is not None:
        from .profile_db import device_tag
        dev = device_tag()
    for i, (p, o) in enumerate(cands):
        key = None
        if db is not None:
            key = db.key(graph.kernel_source(p, o) if graph.family(p, o) != "none" else f"unsupported {p} {o}",
                         warmup, reps, flush_bytes, dev)
            found, val = db.get(key)
            if found:
                costs.append(val)
                continue
        try:
            c = graph.profile(p, o, warmup=warmup, reps=reps, flush_bytes=flush_bytes)
            costs.append(c)
            if db is not None:
                db.put(key, c)
        except KorchError as e:
            if e.code != E_COMPILE:
                raise
            costs.append(None)
            if failures is not None:
                failures.append(((tuple(p), tuple(o)), str(e)[:300]))
        if log and (i + 1) % 50 == 0:
            log(f"profiled {i + 1}/{len(cands)} candidates ({time.time() - t0:.1f} s)")
    if db is not None:
        db.save()
    return costs


def korch_plan(graph, max_prims=64, max_outs=3, warmup=10, reps=100, flush_bytes=512 << 20, log=None,
               extra=(), db=None) -> Choice:
    """Enumerates the supported candidates of ``graph``, profiles them on the
    current device and returns the cheapest ordered plan.  ``extra`` adds
    kernels (e.g. those of hand-written plans) to the candidate set."""
    cands = graph.candidates(max_prims=max_prims, max_outs=max_outs, only_supported=True)
    seen = {(tuple(p), tuple(o)) for p, o in cands}
    for p, o in extra:
        k = (tuple(sorted(p)), tuple(sorted(o)))
        if k not in seen:
            seen.add(k)
            cands.append(k)
    failures = []
    costs = profile_candidates(graph, cands, warmup, reps, flush_bytes, log, failures, db)
    ch = choose(GraphView(graph), cands, costs)
    ch.costs = {(tuple(p), tuple(o)): c for (p, o), c in zip(cands, costs) if c is not None}
    ch.failures = failures
    return ch
