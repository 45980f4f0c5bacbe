"""The measured-cost chooser on the GPU: every supported candidate of each
workload (at the sampled-plan sizes) is profiled, the cheapest ordered plan is
chosen, and that plan must reproduce the unfused float64 oracle and cost no more
than the hand-written plans under the same measured costs."""

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


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("workload", list(SIZES))
def test_chosen_plan(workload):
    from paper_2406_09465_amd import chooser, graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from paper_2406_09465_amd.warm import CHOOSER_LIMITS
    sizes = SIZES[workload]
    w = graphs.build(workload, **sizes)
    print(f"\n[case] {workload} chooser at {sizes}", flush=True)
    hand = {name: w.kernels(name) for name in ("fused", "layered")}
    ch = chooser.korch_plan(w.graph, warmup=3, reps=10, flush_bytes=64 << 20,
                            extra=[k for ks in hand.values() for k in ks], **CHOOSER_LIMITS)
    print(f"[case] {workload}: {ch.candidates} candidates, chosen {len(ch.kernels)} kernels, "
          f"{ch.cost_us:.1f} us", flush=True)
    assert not ch.failures, ch.failures[:2]
    for name, ks in hand.items():
        c = sum(ch.costs[(tuple(sorted(p)), tuple(sorted(o)))] for p, o in ks)
        assert ch.cost_us <= c + 1e-6, (name, c)
    raw, x64 = inputs_f64(workload, **sizes)
    ref = run_unfused(OC.build(workload, **sizes), x64)
    out = PlanRunner(w, kernels=ch.kernels).run(raw)
    for name in w.output_names:
        ok, mx, rel = close(out[name], ref[name], TOL[w.dtype])
        assert ok, f"{workload} chosen plan {ch.kernels}: max err {mx:.3e} rel {rel:.3e}"


@pytest.mark.parametrize("workload", ["attention", "sra", "linattn", "conv"])
def test_chosen_plan_of_transformed_graph(workload):
    """Orchestration of the rewritten primitive graph (Section 3 transformations):
    the chosen plan must reproduce the oracle of the original graph."""
    from paper_2406_09465_amd import chooser, graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from paper_2406_09465_amd.warm import CHOOSER_LIMITS
    sizes = SIZES[workload]
    w, napp = graphs.rewritten(graphs.build(workload, **sizes))
    assert napp > 0
    print(f"\n[case] {workload} transformed graph at {sizes}", flush=True)
    ch = chooser.korch_plan(w.graph, warmup=3, reps=10, flush_bytes=64 << 20, **CHOOSER_LIMITS)
    print(f"[case] {workload}: {ch.candidates} candidates, chosen {len(ch.kernels)} kernels, {ch.cost_us:.1f} us",
          flush=True)
    raw, x64 = inputs_f64(workload, **sizes)
    ref = run_unfused(OC.build(workload, **sizes), x64)
    out = PlanRunner(w, kernels=ch.kernels).run(raw)
    for name in w.output_names:
        ok, mx, rel = close(out[name], ref[name], TOL[w.dtype])
        assert ok, f"{workload} transformed plan {ch.kernels}: max err {mx:.3e} rel {rel:.3e}"


@pytest.mark.parametrize("workload", ["attention", "mlp", "sra", "linattn"])
def test_layout_variant_plans(workload):
    """Layout as a plan variable: on the graph with a transposed-layout variant
    of every computed product operand, seeded random valid plans (which
    materialize some operands transposed) and the measured-cost choice both
    reproduce the oracle of the original graph."""
    from paper_2406_09465_amd import chooser, graphs, search
    from paper_2406_09465_amd._abi import RW_LAYOUT_VARIANTS
    from paper_2406_09465_amd.runner import PlanRunner
    from paper_2406_09465_amd.warm import CHOOSER_LIMITS, SAMPLED
    sizes = SIZES[workload]
    assert SAMPLED[workload][0] == sizes
    w, napp = graphs.rewritten(graphs.build(workload, **sizes), RW_LAYOUT_VARIANTS)
    assert napp > 0
    raw, x64 = inputs_f64(workload, **sizes)
    ref = run_unfused(OC.build(workload, **sizes), x64)
    _, n, seed = SAMPLED[workload]
    plans = search.sampled_plans(w.graph, n, seed)
    print(f"\n[case] {workload} layout variants at {sizes}", flush=True)
    ch = chooser.korch_plan(w.graph, warmup=3, reps=10, flush_bytes=64 << 20, **CHOOSER_LIMITS)
    assert not ch.failures, ch.failures[:2]
    for i, ks in enumerate(plans + [ch.kernels]):
        print(f"[case] {workload} layout plan {i}: {len(ks)} kernels", flush=True)
        out = PlanRunner(w, kernels=ks).run(raw)
        for name in w.output_names:
            ok, mx, rel = close(out[name], ref[name], TOL[w.dtype])
            assert ok, f"{workload} layout plan {i} {ks}: max err {mx:.3e} rel {rel:.3e}"
