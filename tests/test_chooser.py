"""The measured-cost chooser (Section 4.2 with Algorithm 1) against an
exhaustive search of the binary program on small graphs, and against the
hand-written plans of the five workloads under random cost tables.  No GPU: the
costs are synthetic, so these tests check the optimization, not the profiler."""

import itertools
import random

import pytest

from oracle import configs as OC
from oracle.graph import Graph as OGraph
from oracle.orchestration import plan_is_valid
from paper_2406_09465_amd import _abi as K
from paper_2406_09465_amd import chooser, graphs
from paper_2406_09465_amd.search import GraphView


def diamond():
    """x -> a=exp -> {b=neg, c=tanh} -> d=add, plus a reshape view of c;
    outputs d and the view of c (4 primitives that need a kernel)."""
    g = K.Graph()
    og = OGraph()
    x = g.input("f32", (4, 8))
    og.input("x", (4, 8))
    ops = [("exp", [x], {}), ("neg", [1], {}), ("tanh", [1], {}), ("add", [2, 3], {}),
           ("reshape", [3], {"shape": (32,)})]
    for op, ins, at in ops:
        g.op(op, ins, "f32", **at)
        og.op(op, ins, **at)
    for o in (4, 5):
        g.output(o)
        og.output(o)
    g.finalize()
    return g, og


def restricted_candidates(g, rng, size=18):
    """A random subset of the candidates that always holds the one-primitive
    kernels (so that a valid plan exists)."""
    cands = g.candidates(max_prims=16, max_outs=3, only_supported=False)
    singles = [c for c in cands if len(c[0]) == 1 and c[1] == c[0]]
    rest = [c for c in cands if c not in singles]
    return singles + rng.sample(rest, size - len(singles))


def brute_force(view, og, cands, costs, max_kernels):
    """Minimum total cost over kernel subsets satisfying the output and
    dependency constraints that admit an execution order (checked by the
    oracle's plan validator on a greedy order)."""
    best = None
    idx = [i for i, c in enumerate(costs) if c is not None]
    for r in range(1, max_kernels + 1):
        for sub in itertools.combinations(idx, r):
            # greedy order: repeatedly run any kernel whose inputs exist
            avail = set(view.inputs)

            def ok(u):
                return u in avail or (view.op[u] == "reshape" and ok(view.ins[u][0]))
            order, rest = [], list(sub)
            while rest:
                ready = [i for i in rest if all(ok(u) for u in view.external(cands[i][0]))]
                if not ready:
                    break
                i = ready[0]
                order.append(i)
                rest.remove(i)
                avail |= set(cands[i][1])
            if rest:
                continue
            plan = [(list(cands[i][0]), list(cands[i][1])) for i in order]
            if not plan_is_valid(og, plan)[0]:
                continue
            c = sum(costs[i] for i in sub)
            if best is None or c < best:
                best = c
    return best


@pytest.mark.parametrize("seed", range(6))
def test_chooser_matches_exhaustive_program(seed):
    """Every kernel of an optimal plan adds an output that is needed (with
    positive costs a kernel that does not is removable), so an optimum has at
    most as many kernels as primitives that are not views: 4 here."""
    g, og = diamond()
    view = GraphView(g)
    rng = random.Random(seed)
    cands = restricted_candidates(g, rng)
    costs = [rng.uniform(1.0, 10.0) for _ in cands]
    ch = chooser.choose(view, cands, costs)
    assert plan_is_valid(og, ch.kernels)[0]
    assert ch.cost_us == pytest.approx(brute_force(view, og, cands, costs, 4))


def test_chooser_uses_redundancy_when_cheaper():
    """If materializing `a` and multi-output kernels are both expensive, the
    optimum recomputes `a` inside two kernels ({a,c}->c and {a,b}->b, then d)."""
    g, og = diamond()
    view = GraphView(g)
    cands = [c for c in g.candidates(max_prims=16, max_outs=3, only_supported=False) if len(c[0]) <= 3]
    costs = []
    for p, o in cands:
        c = 1.0 + 0.1 * len(p)
        if 1 in o:
            c += 50.0   # materializing `a` is expensive
        c += 20.0 * (len(o) - 1)
        costs.append(c)
    ch = chooser.choose(view, cands, costs)
    assert plan_is_valid(og, ch.kernels)[0]
    assert all(1 not in o for _, o in ch.kernels)
    covered = [set(p) for p, _ in ch.kernels]
    assert sum(1 in p for p in covered) >= 2   # `a` is computed by more than one kernel


@pytest.mark.parametrize("workload", ["attention", "mlp", "sra", "conv", "linattn", "instnorm"])
def test_chooser_never_worse_than_hand_plans(workload):
    w = graphs.build(workload)
    g = w.graph
    view = GraphView(g)
    hand = {name: w.kernels(name) for name in ("fused", "layered")}
    hand["unfused"] = [([v], [v]) for v in sorted(view.op) if view.op[v] not in ("input", "reshape")]
    extra = [k for ks in hand.values() for k in ks]
    cands = g.candidates(max_prims=64, max_outs=3, only_supported=True)
    seen = {(tuple(p), tuple(o)) for p, o in cands}
    for p, o in extra:
        key = (tuple(sorted(p)), tuple(sorted(o)))
        if key not in seen:
            seen.add(key)
            cands.append(key)
    rng = random.Random(11)
    costs = [rng.uniform(1.0, 10.0) for _ in cands]
    table = {(tuple(p), tuple(o)): c for (p, o), c in zip(cands, costs)}
    ch = chooser.choose(view, cands, costs)
    assert plan_is_valid(OC.build(workload), ch.kernels)[0]
    for name, ks in hand.items():
        c = sum(table[(tuple(sorted(p)), tuple(sorted(o)))] for p, o in ks)
        assert ch.cost_us <= c + 1e-9, name


def test_chooser_minimizes_launches_under_uniform_cost():
    """With every kernel costing the same, the optimum is a plan with the fewest
    kernels: attention is one supported kernel."""
    w = graphs.build("attention")
    cands = w.graph.candidates(max_prims=64, max_outs=3, only_supported=True)
    ch = chooser.choose(GraphView(w.graph), cands, [1.0] * len(cands))
    assert len(ch.kernels) == 1 and ch.cost_us == 1.0
