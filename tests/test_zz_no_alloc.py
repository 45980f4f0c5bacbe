"""korch_plan_execute_noalloc (workspace and hand-off counters in the library's
static device scratch, for callers that cannot allocate) against
korch_plan_execute with a caller workspace: the same kernels on the same
inputs give the same bits.

Each case runs two plans in a row through the allocation-free call, the
second on a smaller input, so the second call finds the first call's data
(and counters) in the shared scratch.  The workloads with cross-workgroup
hand-offs (split-K, column reductions) exercise the counter clearing.
"""

import numpy as np
import pytest

from synthetic import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# (workload, plan, first sizes, second smaller sizes)
CASES = [
    ("mlp", "fused", {}, dict(m=300, d=96, h=200)),
    ("linattn", "fused", {}, dict(heads=3, n=300, d=16)),
    ("sra", "fused", {}, dict(hh=40, ww=24, c=16, r=8)),
    ("instnorm", "fused", {}, dict(hh=13, ww=11, c=24)),
    ("conv", "fused", {}, dict(hh=37, ww=29, cin=8, cout=24)),
]


@pytest.fixture(scope="module", autouse=True)

def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _bits(t):
    it = torch.int32 if t.element_size() == 4 else torch.int16
    return t.view(it).cpu().numpy()


def _run_both(workload, plan, sizes):
    """Outputs of korch_plan_execute (caller workspace), then of
    korch_plan_execute_noalloc into fresh buffers, as raw bits."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd._abi import pointer_array
    from paper_2406_09465_amd.runner import PlanRunner
    w = graphs.build(workload, **sizes)
    r = PlanRunner(w, plan)
    r.set_inputs(W.inputs(workload, **sizes))
    r.launch()
    torch.cuda.synchronize()
    ref = [_bits(t) for t in r.outs]
    outs = [torch.full_like(t, float("nan")) for t in r.outs]
    s = torch.cuda.current_stream()
    r.plan.execute_noalloc(pointer_array([t.data_ptr() for t in r.ins]),
                           pointer_array([t.data_ptr() for t in outs]), s.cuda_stream)
    torch.cuda.synchronize()
    return r, ref, [_bits(t) for t in outs]


@pytest.mark.parametrize("workload,plan,big,small", CASES, ids=[c[0] for c in CASES])

def test_noalloc_matches_execute_twice(workload, plan, big, small):
    for sizes in (big, small):
        print(f"\n[case] noalloc {workload} {plan} {sizes}", flush=True)
        r, ref, got = _run_both(workload, plan, sizes)
        for a, b in zip(ref, got):
            assert a.shape == b.shape
            assert np.array_equal(a, b), f"{workload} {sizes}: {np.count_nonzero(a != b)} elements differ"


def test_noalloc_does_not_allocate():
    """Repeated allocation-free calls leave the device's free memory unchanged."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd._abi import pointer_array
    from paper_2406_09465_amd.runner import PlanRunner
    print("\n[case] noalloc free memory", flush=True)
    w = graphs.build("linattn")
    r = PlanRunner(w, "fused")
    r.set_inputs(W.inputs("linattn"))
    ins = pointer_array([t.data_ptr() for t in r.ins])
    outs = pointer_array([t.data_ptr() for t in r.outs])
    st = torch.cuda.current_stream().cuda_stream
    r.plan.execute_noalloc(ins, outs, st)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for _ in range(20):
        r.plan.execute_noalloc(ins, outs, st)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0


def test_noalloc_rejects_a_plan_beyond_the_static_scratch():
    """The unfused MLP plan needs 48 MiB of workspace: refused, nothing launched."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd._abi import KorchError, pointer_array
    from paper_2406_09465_amd.runner import PlanRunner
    print("\n[case] noalloc oversized plan", flush=True)
    w = graphs.build("mlp")
    r = PlanRunner(w, "unfused")
    assert r.ws_bytes > 32 << 20
    r.set_inputs(W.inputs("mlp"))
    out = torch.zeros_like(r.outs[0])
    with pytest.raises(KorchError) as e:
        r.plan.execute_noalloc(pointer_array([t.data_ptr() for t in r.ins]), pointer_array([out.data_ptr()]),
                               torch.cuda.current_stream().cuda_stream)
    assert e.value.code == -22 and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(out)) == 0
