"""Orchestration experiments on the GPU.

  python -m paper_2406_09465_amd.experiments shapes --out profiles/chooser_shapes.md

  python -m paper_2406_09465_amd.experiments layouts --out profiles/chooser_layouts.md

``shapes``: the measured-cost chooser on one workload at several sizes.  The
paper observes that the best orchestration of the same subgraph changes with its
shape (a memory-bound subgraph fused into one kernel at batch 1 but split into
several at batch 16, Section 6): the chosen plan here is recorded per size with
its number of kernels, its predicted cost (sum of measured kernel latencies)
and the cost of fusing everything the families allow into the fewest kernels.

``layouts``: data layout as a plan variable (the extension of the
orchestration formulation in Section 8).  Each workload's graph gets a
transposed-layout variant of every computed operand of a product
(``RW_LAYOUT_VARIANTS``); the chooser then decides, per tensor, in which layout
it is materialized and how each consumer reads it.  Recorded per workload: the
chosen plan on the original and on the variant graph, and, for each variant,
the cheapest plan that stores that tensor only in the transposed layout (its
row-major kernels removed), i.e. what the layout choice is weighed against.
"""

from __future__ import annotations

import argparse
import concurrent.futures as cf
import multiprocessing as mp
import os
import time

from . import chooser, graphs
from .search import GraphView

SWEEPS = {
    "attention": [dict(n=n, d=64) for n in (32, 64, 128, 256)],
    "linattn": [dict(heads=16, n=n, d=16) for n in (256, 1024, 4096, 16384)],
    "mlp": [dict(m=m, d=768, h=3072) for m in (128, 512, 2048, 8192)],
    "sra": [dict(hh=h, ww=h, c=64, r=8) for h in (32, 64, 128, 256)],
    "instnorm": [dict(hh=h, ww=h, c=32) for h in (28, 56, 112, 224, 448)],
}
LIMITS = dict(max_prims=64, max_outs=3)


def _compile_share(args):
    workload, sizes, part, parts = args
    w = graphs.build(workload, **sizes)
    w2, napp = graphs.rewritten(w)
    bad = 0
    for g in ([w.graph, w2.graph] if napp else [w.graph]):  # the transformed graph too, where a rule applies
        cands = g.candidates(only_supported=True, **LIMITS)
        for c in cands[part::parts]:
            try:
                g.compile_candidate(*c)
            except Exception:
                bad += 1
    return bad


def precompile(jobs, processes=None):
    """Compiles the supported candidates of every (workload, sizes) in ``jobs``
    in worker processes (hipRTC serializes compiles inside one process)."""
    procs = processes or min(16, os.cpu_count() or 1)
    tasks = [(w, sz, i, procs) for w, sz in jobs for i in range(procs)]
    with cf.ProcessPoolExecutor(max_workers=procs, mp_context=mp.get_context("spawn")) as ex:
        return sum(ex.map(_compile_share, tasks))


def fewest_kernels(view, cands, costs):
    """The plan with the fewest kernels (ties broken by measured cost)."""
    big = 1e6
    c2 = [None if c is None else big + c for c in costs]
    ch = chooser.choose(view, cands, c2)
    n = len(ch.kernels)
    return n, ch.cost_us - n * big


def shapes(workload, out, warmup=10, reps=100):
    jobs = [(workload, sz) for sz in SWEEPS[workload]]
    t0 = time.time()
    precompile(jobs)
    lines = [f"# Measured-cost orchestration of `{workload}` across sizes", "",
             "Command:", "", "```", f"python -m paper_2406_09465_amd.experiments shapes --workload {workload} "
             f"--out {out}", "```", "",
             f"Candidates compiled in {time.time() - t0:.0f} s. Costs are medians of {reps} launches after "
             f"{warmup} warm-up launches, each timed by its own dispatch after a read of 512 MiB (cold caches) and "
             "a read of its computed inputs (cache-resident, as a producing kernel leaves them).", "",
             "The last column is the cheapest plan of the graph after the primitive-graph transformations "
             "(`korch_graph_rewrite`, all rules), where any applies; the chooser of the bench keeps the cheaper graph.", "",
             "| sizes | candidates | chosen kernels | chosen cost (us) | fewest kernels | their cost (us) | chosen plan | "
             "transformed graph: cost (us), kernels |",
             "|---|---|---|---|---|---|---|---|"]
    for sz in SWEEPS[workload]:
        w = graphs.build(workload, **sz)
        cands = w.graph.candidates(only_supported=True, **LIMITS)
        costs = chooser.profile_candidates(w.graph, cands, warmup, reps)
        view = GraphView(w.graph)
        ch = chooser.choose(view, cands, costs)
        nf, cf_ = fewest_kernels(view, cands, costs)
        names = {v: k for k, v in w.ids.items()}
        plan = " ; ".join("{" + ",".join(names[v] for v in o) + "}" for _, o in ch.kernels)
        w2, napp = graphs.rewritten(w)
        rw = "none applies"
        if napp:
            ch2 = chooser.korch_plan(w2.graph, **LIMITS, warmup=warmup, reps=reps)
            rw = f"{ch2.cost_us:.2f}, {len(ch2.kernels)}"
        lines.append(f"| {sz} | {sum(c is not None for c in costs)} | {len(ch.kernels)} | {ch.cost_us:.2f} | {nf} | "
                     f"{cf_:.2f} | {plan} | {rw} |")
        print(lines[-1], flush=True)
    open(out, "w").write("\n".join(lines) + "\n")


def layouts(out, workloads=None, warmup=10, reps=100):
    from ._abi import RW_LAYOUT_VARIANTS
    from .warm import LAYOUT_WORKLOADS
    wls = list(workloads or LAYOUT_WORKLOADS)
    lines = ["# Data layout as a plan variable", "", "Command:", "", "```",
             f"python -m paper_2406_09465_amd.experiments layouts --out {out}", "```", "",
             f"Full-size workloads; costs are medians of {reps} launches after {warmup} warm-up launches, each timed "
             "by its own dispatch after a read of 512 MiB (cold caches) and a read of its computed inputs.  `x^T` is tensor x stored with its last two axes swapped.", "",
             "| workload | original graph (us, kernels) | variant graph (us, kernels) | layouts chosen | "
             "cheapest plan storing only x^T, per variant (us) |", "|---|---|---|---|---|"]
    for wl in wls:
        w = graphs.build(wl)
        base = chooser.korch_plan(w.graph, **LIMITS, warmup=warmup, reps=reps)
        w2, n = graphs.rewritten(w, RW_LAYOUT_VARIANTS)
        g = w2.graph
        ch = chooser.korch_plan(g, **LIMITS, warmup=warmup, reps=reps)
        view = GraphView(g)
        # variant pairs: x -> x^T -> (x^T)^T
        pairs = []
        for v in range(g.num_nodes()):
            if view.op[v] == "transpose" and view.op[view.ins[v][0]] != "transpose":
                nxt = [c for c in range(g.num_nodes()) if view.op[c] == "transpose" and view.ins[c] == [v]]
                if nxt:
                    pairs.append((view.ins[v][0], v))
        names = {}
        orig_names = {v: k for k, v in w.ids.items()}
        for x, xt in pairs:
            op, _, shape = g.node_info(x)
            names[x] = f"{op}{list(shape)}"
            names[xt] = names[x] + "^T"
        chosen_t = sorted({names[o] for _, outs in ch.kernels for o in outs if o in names and o in dict(pairs).values()})
        forced = []
        cands = list(ch.costs)
        for x, xt in pairs:
            costs = [None if x in o else ch.costs[(p, o)] for p, o in cands]
            try:
                f = chooser.choose(view, cands, costs)
                forced.append(f"{names[xt]}: {f.cost_us:.2f}")
            except RuntimeError:
                forced.append(f"{names[xt]}: no plan")
        lines.append(f"| {wl} | {base.cost_us:.2f}, {len(base.kernels)} | {ch.cost_us:.2f}, {len(ch.kernels)} | "
                     f"{', '.join(chosen_t) or 'none (all row-major)'} | {'; '.join(forced)} |")
        print(lines[-1], flush=True)
    open(out, "w").write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    s = sub.add_parser("shapes")
    s.add_argument("--workload", default="attention", choices=list(SWEEPS))
    s.add_argument("--out", required=True)
    lo = sub.add_parser("layouts")
    lo.add_argument("--out", required=True)
    lo.add_argument("--workloads", nargs="*", default=None)
    a = ap.parse_args()
    if a.mode == "shapes":
        shapes(a.workload, a.out)
    else:
        layouts(a.out, a.workloads)


if __name__ == "__main__":
    main()
