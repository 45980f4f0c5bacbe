"""GPU parity of seeded random orchestration plans, and the kernel profiler.

Every valid plan -- any grouping of primitives into supported convex kernels,
with redundant execution and pruning -- must reproduce the unfused float64
oracle within the dtype tolerance (fusion changes cost, not the result).
"""

import math

import pytest

from oracle import configs as OC
from oracle.graph import run_unfused
from tests.helpers import TOL, close, inputs_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SIZES = {
    "attention": dict(n=96, d=32),
    "mlp": dict(m=256, d=128, h=192),
    "sra": dict(hh=32, ww=32, c=32, r=8),
    "conv": dict(hh=24, ww=20, cin=16, cout=32),
    "linattn": dict(heads=4, n=512, d=16),
    "instnorm": dict(hh=40, ww=36, c=16),
}
N_PLANS = 6
SEED = 7


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("workload", list(SIZES))
def test_sampled_plans(workload):
    from paper_2406_09465_amd import graphs, search
    from paper_2406_09465_amd.runner import PlanRunner
    sizes = SIZES[workload]
    w = graphs.build(workload, **sizes)
    raw, x64 = inputs_f64(workload, **sizes)
    ref = run_unfused(OC.build(workload, **sizes), x64)
    plans = search.sampled_plans(w.graph, N_PLANS, SEED)
    tol = TOL[w.dtype]
    for i, ks in enumerate(plans):
        print(f"\n[case] {workload} sampled plan {i}: {len(ks)} kernels", flush=True)
        out = PlanRunner(w, kernels=ks).run(raw)
        for name in w.output_names:
            ok, mx, rel = close(out[name], ref[name], tol)
            assert ok, f"{workload} plan {i} {ks}: max err {mx:.3e} rel {rel:.3e}"


def test_profiler_times_candidates():
    from paper_2406_09465_amd import graphs
    w = graphs.mlp(**SIZES["mlp"])
    print("\n[case] profiler", flush=True)
    for prims, outs in w.kernels("fused"):
        us = w.graph.profile(prims, outs, warmup=3, reps=10, flush_bytes=64 << 20)
        assert us is not None and math.isfinite(us) and 0.5 < us < 5000.0
    ids = w.ids
    # a kernel no family implements costs infinity (None)
    assert w.graph.profile([ids["var"], ids["ve"], ids["r"], ids["Xh"], ids["Yg"], ids["Y"], ids["H0"]],
                           [ids["H0"]], warmup=1, reps=1) is None


def test_timed_execution_matches_plain_execution():
    """korch_plan_execute_timed launches the same kernels as korch_plan_execute
    (identical bytes) and brackets the timed kernel with the caller's events."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W
    sizes = SIZES["mlp"]
    w = graphs.build("mlp", **sizes)
    print("\n[case] timed execution, mlp layered", flush=True)
    r = PlanRunner(w, "layered")
    r.set_inputs(W.inputs("mlp", **sizes))
    r.launch()
    torch.cuda.synchronize()
    ref = [t.clone() for t in r.outs]
    s = torch.cuda.current_stream()
    for k in range(r.plan.num_kernels()):
        for t in r.outs:
            t.zero_()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        b.record(s)
        r.launch_timed(k, a, b)
        torch.cuda.synchronize()
        assert all(torch.equal(x, y) for x, y in zip(ref, r.outs))
        assert a.elapsed_time(b) > 0.0
        # the same through the pre-bound arguments
        for t in r.outs:
            t.zero_()
        r.bind()
        r.launch_timed_bound(k, a, b)
        torch.cuda.synchronize()
        assert all(torch.equal(x, y) for x, y in zip(ref, r.outs))
        for t in r.outs:
            t.zero_()
        r.launch_bound()
        torch.cuda.synchronize()
        assert all(torch.equal(x, y) for x, y in zip(ref, r.outs))


@pytest.mark.parametrize("workload,plan", [("linattn", "fused"), ("sra", "fused"), ("instnorm", "layered")])
def test_cross_workgroup_handoff_repeats_bitwise(workload, plan):
    """Kernels whose workgroups hand fp32 partials to a last workgroup (split-K,
    column reductions) give identical bytes on every one of many back-to-back
    executions (partials read coherently, fixed combination order)."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W
    print(f"\n[case] {workload} {plan} repeated", flush=True)
    r = PlanRunner(graphs.build(workload), plan)
    r.set_inputs(W.inputs(workload))
    r.launch()
    torch.cuda.synchronize()
    ref = [t.clone() for t in r.outs]
    it = torch.int16 if ref[0].element_size() == 2 else torch.int32
    for _ in range(200):
        for t in r.outs:
            t.zero_()
        r.launch()
        torch.cuda.synchronize()
        assert all(torch.equal(a.view(it), b.view(it)) for a, b in zip(ref, r.outs))


def test_execute_with_events_on_every_kernel():
    """korch_plan_execute_events launches the same kernels as korch_plan_execute
    (identical bytes); events on every kernel give positive durations that lie
    inside the span from the first kernel's start to the last kernel's end, and
    NULL entries are allowed."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W
    sizes = SIZES["mlp"]
    w = graphs.build("mlp", **sizes)
    print("\n[case] per-kernel events, mlp layered", flush=True)
    r = PlanRunner(w, "layered")
    r.set_inputs(W.inputs("mlp", **sizes))
    r.launch()
    torch.cuda.synchronize()
    ref = [t.clone() for t in r.outs]
    s = torch.cuda.current_stream()
    r.bind(s)
    nk = r.plan.num_kernels()
    assert nk >= 2
    st = [torch.cuda.Event(enable_timing=True) for _ in range(nk)]
    en = [torch.cuda.Event(enable_timing=True) for _ in range(nk)]
    for e in st + en:
        e.record(s)
    for t in r.outs:
        t.zero_()
    r.launch_events_bound(r.event_arrays(st, en))
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(ref, r.outs))
    span = st[0].elapsed_time(en[-1])
    durs = [st[k].elapsed_time(en[k]) for k in range(nk)]
    assert all(d > 0.0 for d in durs)
    assert span >= max(durs) and span >= 0.9 * sum(durs)
    for k in range(1, nk):
        assert st[k - 1].elapsed_time(st[k]) >= 0.0  # kernels start in plan order
    # only the first start and the last stop
    a = [st[0]] + [None] * (nk - 1)
    b = [None] * (nk - 1) + [en[-1]]
    for t in r.outs:
        t.zero_()
    r.launch_events_bound(r.event_arrays(a, b))
    torch.cuda.synchronize()
    assert all(torch.equal(x, y) for x, y in zip(ref, r.outs))
    assert st[0].elapsed_time(en[-1]) > 0.0


def test_cache_flush_read_and_write():
    """korch_flush_caches: the read flush leaves its buffer unchanged, the
    write flush overwrites it; both run on the caller's stream."""
    import ctypes as C

    from paper_2406_09465_amd._abi import lib
    print("\n[case] cache flush", flush=True)
    buf = torch.arange(1 << 20, dtype=torch.int32, device="cuda")  # 4 MiB
    ref = buf.clone()
    s = torch.cuda.current_stream()
    nb = buf.numel() * 4
    assert lib.korch_flush_caches(C.c_void_p(buf.data_ptr()), C.c_size_t(nb), 0, C.c_void_p(s.cuda_stream)) == 0
    torch.cuda.synchronize()
    assert torch.equal(buf, ref)
    assert lib.korch_flush_caches(C.c_void_p(buf.data_ptr()), C.c_size_t(nb), 1, C.c_void_p(s.cuda_stream)) == 0
    torch.cuda.synchronize()
    assert not torch.equal(buf, ref)
