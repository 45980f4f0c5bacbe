"""Fused-subgraph latency of one workload's orchestration plan on one MI355X.

One step = one execution of the whole plan (every kernel of the fused
orchestration) on inputs already resident in HBM.  Before every timed step a
read of a 512 MiB device buffer evicts L2 and the Infinity Cache (the
workloads' working sets would otherwise stay cache-resident); the step's latency is the span from
its first kernel's dispatch start to its last kernel's dispatch end, taken by
events attached to those dispatches.  `value` is the median over the timed
steps (p10 / p90 beside it); the same plan back to back without flushes is
reported as `warm`.

Prints ONE JSON line: metric / value (microseconds per step), a roofline
object for the plan's dominant kernel (algorithmic flops or bytes per launch
over its mean launch duration in the timed steps), the measured-cost model's
prediction against the measured step, the unfused plan of the same graph under
the same protocol, and the float64 oracle timed on the host cores on a bounded
sample.

Default workload: transformer MLP block, fp16, X [4096, 768], W1 [768, 3072],
W2 [3072, 768] (the configuration the headline metric is quoted on).
"""

from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fused-subgraph latency (µs) & achieved HBM GB/s or MFMA util vs peak, 1×MI355X"
PEAK = {  # MI355X published peaks
    "hbm_GBs": 8000.0,
    "mfma_f16_TFLOPs": 2500.0,
    "mfma_bf16_TFLOPs": 2500.0,
    "f32_TFLOPs": 157.3,
}
DESCR = {
    "attention": "single-head attention fp32, Q,K,V [128,64]",
    "mlp": "transformer MLP block fp16: LayerNorm, X[4096,768] x W1[768,3072], tanh-GELU, x W2[3072,768], residual",
    "sra": "spatial-reduction attention fp16: 128x128x64 map, 8x8 patch merge 4096->64, LayerNorm, 16384x256 softmax",
    "conv": "conv3x3 NHWC fp16 416x416x32->64 + BatchNorm scale/shift + Mish",
    "linattn": "ReLU linear attention bf16, 16 heads x 4096 tokens x d16",
    "instnorm": "InstanceNorm + ReLU + zero Pad fp16 NHWC 224x224x32 -> 226x226x32",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400,
                    help="timed steps, each preceded by a cache flush and timed from its first kernel's start "
                         "to its last kernel's end")
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="mlp", choices=list(DESCR))
    ap.add_argument("--plan", default="korch",
                    help="korch (profile every candidate kernel on this GPU and run the cheapest valid plan; the "
                         "default) | fused | layered | unfused (hand-written plans)")
    ap.add_argument("--kernels-json", default="",
                    help="run the plan recorded (chosen_plan) in an earlier bench.py output line instead")
    ap.add_argument("--no-rewrite", action="store_true",
                    help="korch plan: do not consider the transformed primitive graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true", help="skip the unfused-plan comparison")
    ap.add_argument("--flush-mib", type=int, default=512,
                    help="MiB streamed through before every timed step to evict L2 and the Infinity Cache")
    ap.add_argument("--flush-write", action="store_true",
                    help="the flush writes its buffer (leaving dirty lines) instead of reading it")
    ap.add_argument("--profile-reps", type=int, default=100, help="timed launches per candidate in the chooser")
    ap.add_argument("--no-profile-db", action="store_true",
                    help="profile every candidate again instead of reusing latencies recorded in the profile database")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target CPU work for the oracle sample")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before timing, run a plain device copy of this many MiB 3 times (PMC byte calibration)")
    return ap.parse_args()


def cpu_baseline(workload, seconds):
    """The float64 oracle (unfused, one primitive at a time) on the host cores."""
    import numpy as np
    from oracle import configs as OC
    from oracle.graph import run_unfused
    from synthetic import storage_to_f64
    from synthetic import workloads as W
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    dt = W.DEFAULT_DTYPE[workload]
    raw = W.inputs(workload)
    x64 = {k: storage_to_f64(v, dt) for k, v in raw.items()}
    g = OC.build(workload)
    times = []
    t_end = time.perf_counter() + seconds
    while True:
        t0 = time.perf_counter()
        run_unfused(g, x64)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() >= t_end and len(times) >= 3:
            break
    med = statistics.median(times)
    return {"value": med * 1e6, "unit": "us", "cores": int(threads), "kind": "oracle",
            "sample": f"{len(times)} full runs of the unfused float64 oracle on the whole workload "
                      f"({sum(times):.1f} s of CPU work); value = median microseconds per run"}


def traffic_from_profiles(kernel_name, source_hash):
    """HBM bytes per launch of the dominant kernel from committed rocprofv3 PMC
    summaries (FETCH_SIZE / WRITE_SIZE), or None if absent or stale."""
    path = os.path.join(ROOT, "profiles", "pmc_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        data = json.load(open(path))
        rec = data["kernels"].get(kernel_name)  # "<workload>/<kernel name>"
        if not rec or rec.get("source_hash") != source_hash:
            return None
        return rec["hbm_bytes_per_launch"]
    except Exception:
        return None


def pct(xs):
    """n, p10, median, p90 (microseconds) of a sample."""
    ys = sorted(xs)

    def q(f):
        return round(ys[min(len(ys) - 1, int(f * (len(ys) - 1) + 0.5))], 3)
    return {"n": len(ys), "p10_us": q(0.1), "median_us": round(statistics.median(ys), 3), "p90_us": q(0.9)}


class Flush:
    """Cold-cache precondition: korch_flush_caches over a device buffer (a
    read by default; a write with write=True), enqueued on the stream."""

    def __init__(self, mib, stream, write=False):
        import ctypes as C

        import torch

        from paper_2406_09465_amd._abi import lib
        self.buf = torch.empty(max(1, mib) << 20, dtype=torch.uint8, device="cuda")
        self.args = (C.c_void_p(self.buf.data_ptr()), C.c_size_t(self.buf.numel()), C.c_int32(1 if write else 0),
                     C.c_void_p(stream.cuda_stream))
        self.lib = lib

    def __call__(self):
        rc = self.lib.korch_flush_caches(*self.args)
        if rc:
            from paper_2406_09465_amd._abi import check
            check(rc)


def timed_steps(r, steps, flush, stream):
    """Runs `steps` executions of the bound plan of runner `r` on `stream`.
    Before each one, when `flush` (a Flush) is given, it runs, outside the
    measured span.  Every execution carries an event on the start of its first
    kernel's dispatch and one on the end of every kernel's dispatch
    (end-of-dispatch events add nothing to the span; a start event on a later
    kernel adds a few microseconds, so none is used).  Returns the spans (first
    kernel's start to last kernel's end, us), each kernel's duration in every
    execution (us; kernel k > 0: from the end of kernel k - 1 to its own end,
    i.e. including the dispatch gap in front of it), and the wall time of the
    loop (s)."""
    import torch
    nk = r.plan.num_kernels()
    recs = []
    for _ in range(steps):
        st = [torch.cuda.Event(enable_timing=True)] + [None] * (nk - 1)
        en = [torch.cuda.Event(enable_timing=True) for _ in range(nk)]
        for e in st[:1] + en:
            e.record(stream)  # creates the underlying event
        recs.append((st, en, r.event_arrays(st, en)))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _, _, arr in recs:
        if flush is not None:
            flush()
        r.launch_events_bound(arr)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    spans = [st[0].elapsed_time(en[nk - 1]) * 1e3 for st, en, _ in recs]
    per = [[(st[0] if k == 0 else en[k - 1]).elapsed_time(en[k]) * 1e3 for st, en, _ in recs] for k in range(nk)]
    return {"spans": spans, "per_kernel": per, "wall_s": wall}


# Relative cost margin a transformed graph's plan must beat the original's by.
TIE_MARGIN = 0.02


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on exactly one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import hashlib

    import torch

    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W

    torch.cuda.set_device(0)
    if args.flush_write:
        os.environ["KORCH_FLUSH_WRITE"] = "1"  # the profiler's flush then writes too
    w = graphs.build(args.workload)
    chosen = None
    if args.kernels_json:
        d = json.loads(open(args.kernels_json).read().strip().splitlines()[-1])
        chosen = d["chosen_plan"]
        w, ks = graphs.plan_from_record(w, chosen)
        r = PlanRunner(w, kernels=ks)
    elif args.plan == "korch":
        # Orchestration over the primitive graph and over its transformed
        # version (Section 3 rewrites); the cheaper measured plan runs.
        from paper_2406_09465_amd import chooser
        from paper_2406_09465_amd._abi import RW_ALL, RW_LAYOUT_VARIANTS
        from paper_2406_09465_amd.warm import CHOOSER_LIMITS, LAYOUT_WORKLOADS
        t0 = time.time()
        hand = [k for name in ("fused", "layered") for k in w.kernels(name)]
        db = None
        if not args.no_profile_db:
            from paper_2406_09465_amd.profile_db import ProfileDB
            db = ProfileDB()
        prof = dict(warmup=10, reps=args.profile_reps, flush_bytes=args.flush_mib << 20, db=db)
        ch = chooser.korch_plan(w.graph, extra=hand, **prof, **CHOOSER_LIMITS)
        best, rules, w0 = ch, 0, w
        alt = lay = None
        if not args.no_rewrite:
            # the transformed graph, and the graph with layout variants of the
            # computed product operands (layout as a plan variable)
            for rr in (RW_ALL, RW_LAYOUT_VARIANTS):
                if rr == RW_LAYOUT_VARIANTS and args.workload not in LAYOUT_WORKLOADS:
                    continue
                w2, napp = graphs.rewritten(w0, rr)
                if not napp:
                    continue
                c2 = chooser.korch_plan(w2.graph, **prof, **CHOOSER_LIMITS)
                if rr == RW_ALL:
                    alt = c2
                else:
                    lay = c2
                # a transformed graph replaces the original only when its plan
                # is cheaper by more than the run-to-run spread of the profiled
                # costs (about 2 %), so near-ties keep the same kernels
                if c2.cost_us < best.cost_us * (1.0 - TIE_MARGIN):
                    best, rules, w = c2, rr, w2
        chosen = graphs.plan_record(w, best.kernels, rules)
        chosen.update({"predicted_us": round(best.cost_us, 3), "candidates": best.candidates,
                       "search_states": best.states, "original_graph_us": round(ch.cost_us, 3),
                       "rewritten_graph_us": round(alt.cost_us, 3) if alt else None,
                       "layout_graph_us": round(lay.cost_us, 3) if lay else None,
                       "choose_seconds": round(time.time() - t0, 1),
                       "profile_db": {"path": db.path, "hits": db.hits, "new": db.new} if db else None})
        r = PlanRunner(w, kernels=best.kernels)
    else:
        r = PlanRunner(w, args.plan)
    r.set_inputs(W.inputs(args.workload))
    nk = r.plan.num_kernels()
    stream = torch.cuda.current_stream()

    if args.calib_copy_mib:
        # A plain streaming kernel of known traffic for the byte counters:
        # dst = src + 1 reads and writes exactly n bytes each (uint8).
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.add(src, 1, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # warm-up, then the timed region: exactly `steps` plan executions.  Before
    # every step a read of `flush_mib` MiB of a scratch buffer (outside the
    # measured span) evicts L2 and the Infinity Cache, so the step reads its
    # inputs from HBM.  A step's
    # latency is the span from its first kernel's dispatch start to its last
    # kernel's dispatch end, taken by events that the library attaches to those
    # dispatches (no marker packets); end-of-dispatch events on every kernel
    # give the per-kernel durations and the dominant kernel's launch time.
    for _ in range(args.warmup):
        r.launch()
    r.bind(stream)
    flush = Flush(args.flush_mib, stream, args.flush_write) if args.flush_mib else None
    res = timed_steps(r, args.steps, flush, stream)
    spans = res["spans"]
    per = res["per_kernel"]
    dom = max(range(nk), key=lambda k: statistics.median(per[k]))
    dom_us = statistics.mean(per[dom])
    value_us = statistics.median(spans)
    dist = pct(spans)
    if args.steps < 200:
        # the timing protocol's sample size: more flushed steps outside the
        # timed region, for the distribution only
        more = timed_steps(r, 200 - args.steps, flush, stream)["spans"]
        d2 = pct(spans + more)
        dist["n200"] = {k_: d2[k_] for k_ in ("n", "p10_us", "median_us", "p90_us")}
    # the other cold precondition: a flush that writes (the step's misses then
    # also write back the flush buffer's dirty lines)
    other = None
    if args.flush_mib:
        oflush = Flush(args.flush_mib, stream, not args.flush_write)
        o = timed_steps(r, 100, oflush, stream)
        other = dict(pct(o["spans"]), flush="write" if not args.flush_write else "read",
                     kernels_median_us=[round(statistics.median(x), 3) for x in o["per_kernel"]])
        del oflush
    # the same plan back to back without flushes (warm caches)
    warm = timed_steps(r, max(args.steps, 50), None, stream)
    warm_d = pct(warm["spans"])
    warm_d["back_to_back_us_per_step"] = round(warm["wall_s"] * 1e6 / max(args.steps, 50), 3)
    warm_d["note"] = "no flush: inputs and weights resident in L2 / Infinity Cache"

    fam, abytes, aflops = r.plan.kernel_info(dom)
    name = r.plan.kernel_name(dom)
    src_hash = hashlib.sha256(r.plan.kernel_source(dom).encode()).hexdigest()[:16]
    # bound by the roofline: above the ridge (peak flops of the dtype / HBM
    # bandwidth) the kernel is compute-bound, below it memory-bound
    peak = PEAK["f32_TFLOPs"] if w.dtype == "f32" else PEAK[f"mfma_{w.dtype}_TFLOPs"]
    ridge = peak * 1e12 / (PEAK["hbm_GBs"] * 1e9)
    if aflops > 0 and fam in ("gemm", "conv", "attention", "splitk") and aflops / max(abytes, 1) > ridge:
        achieved = aflops / (dom_us * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4)}
    else:
        achieved = abytes / (dom_us * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK["hbm_GBs"], "unit": "GB/s",
                "frac": round(achieved / PEAK["hbm_GBs"], 4)}
    roof["traffic"] = traffic_from_profiles(f"{args.workload}/{name}", src_hash)
    roof["kernel"] = name
    roof["kernel_us"] = round(dom_us, 3)
    roof["timed_launches"] = len(per[dom])
    roof["alg_bytes"] = abytes
    roof["alg_flops"] = aflops
    roof["source_hash"] = src_hash

    # context floors (same run, same stream): a launch of a one-element kernel,
    # and a device copy moving the plan's algorithmic bytes per step (half read,
    # half written), each timed back to back
    def per_launch_us(fn, n=200):
        fn()
        a_, b_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a_.record(stream)
        for _ in range(n):
            fn()
        b_.record(stream)
        torch.cuda.synchronize()
        return a_.elapsed_time(b_) * 1e3 / n
    step_bytes = sum(r.plan.kernel_info(k)[1] for k in range(nk))
    one = torch.zeros(1, device="cuda")
    csrc = torch.empty(max(16, int(step_bytes) // 2), dtype=torch.uint8, device="cuda")
    cdst = torch.empty_like(csrc)
    floors = {"empty_kernel_us": round(per_launch_us(lambda: one.add_(1.0)), 3),
              "copy_us": round(per_launch_us(lambda: cdst.copy_(csrc)), 3), "copy_bytes_moved": 2 * csrc.numel()}
    del one, csrc, cdst

    # context: the unfused plan of the same primitive graph (one kernel per
    # primitive, contiguous reshapes as views), same inputs, same protocol
    unfused = None
    if not args.no_unfused:
        ru = PlanRunner(graphs.build(args.workload), "unfused")
        ru.set_inputs(W.inputs(args.workload))
        for _ in range(5):
            ru.launch()
        ru.bind(stream)
        n_unf = max(20, args.steps // 2)
        uf = timed_steps(ru, n_unf, flush, stream)
        uw = timed_steps(ru, n_unf, None, stream)
        unfused = {"us_per_step": round(statistics.median(uf["spans"]), 3), "flushed": pct(uf["spans"]),
                   "warm": pct(uw["spans"]), "kernels": ru.plan.num_kernels(), "steps": n_unf}
        del ru
    del flush

    kernels = []
    for k in range(nk):
        f, b, fl = r.plan.kernel_info(k)
        kernels.append({"name": r.plan.kernel_name(k), "family": f, "us": round(statistics.median(per[k]), 3),
                        "warm_us": round(statistics.median(warm["per_kernel"][k]), 3),
                        "alg_bytes": b, "alg_flops": fl})

    out = {
        "metric": METRIC,
        "value": round(value_us, 3),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(value_us * 1e-3, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": DESCR[args.workload], "plan": "recorded" if args.kernels_json else args.plan,
                   "kernels": nk},
        "timing": dict(dist, protocol=f"each step after a {args.flush_mib} MiB "
                                         f"{'write' if args.flush_write else 'read'} of a scratch buffer (outside the "
                                         "span; evicts L2 and the Infinity Cache); span = first kernel's dispatch start "
                                         "to last kernel's dispatch end; value = median",
                       wall_s_with_flushes=round(res["wall_s"], 4)),
        "timing_other_flush": other,
        "warm": warm_d,
        "roofline": roof,
        "unfused": unfused,
        "floors": floors,
        "kernels": kernels,
    }
    if chosen:
        out["chosen_plan"] = chosen
        if chosen.get("predicted_us"):
            # the cost model (sum of the kernels' profiled latencies) against
            # the measured flushed step
            out["cost_model"] = {"predicted_us": chosen["predicted_us"], "measured_us": round(value_us, 3),
                                 "sum_kernel_medians_us": round(sum(statistics.median(p_) for p_ in per), 3),
                                 "predicted_over_measured": round(chosen["predicted_us"] / value_us, 4)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
