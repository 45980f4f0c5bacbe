"""GPU parity: every plan of every workload against the float64 oracle.

The HIP path (generated gfx950 kernels behind the C ABI) and the oracle run on
the same seeded, dtype-rounded inputs.  Pass rule per element:
|gpu - ref| <= tol*|ref| + tol*max|ref|, with tol = 1e-5 (fp32), 2e-2 (fp16),
3e-2 (bf16).  Full workload sizes are compared on every element (the oracle
finishes them in seconds); small ragged sizes exercise partial tiles.
"""

import numpy as np
import pytest

from oracle import configs as OC
from oracle.graph import run_unfused
from tests.helpers import TOL, close, close_elementwise, inputs_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

FULL = {
    "attention": {},
    "mlp": {},
    "sra": {},
    "conv": {},
    "linattn": {},
    "instnorm": {},
}
RAGGED = {
    "attention": dict(n=50, d=24),
    "mlp": dict(m=300, d=96, h=200),
    "sra": dict(hh=40, ww=24, c=16, r=8),
    "conv": dict(hh=37, ww=29, cin=8, cout=24),
    "linattn": dict(heads=3, n=300, d=16),
    "instnorm": dict(hh=13, ww=11, c=24),
}
PLANS = ["unfused", "layered", "fused"]

_ref_cache = {}


def reference(workload, sizes):
    key = (workload, tuple(sorted(sizes.items())))
    if key not in _ref_cache:
        raw, x64 = inputs_f64(workload, **sizes)
        ref = run_unfused(OC.build(workload, **sizes), x64)
        _ref_cache.clear()
        _ref_cache[key] = (raw, ref)
    return _ref_cache[key]


def run_plan(workload, sizes, plan):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    w = graphs.build(workload, **sizes)
    raw, ref = reference(workload, sizes)
    r = PlanRunner(w, plan)
    out = r.run(raw)
    return w, r, raw, ref, out


def check(workload, w, out, ref):
    tol = TOL[w.dtype]
    for name in w.output_names:
        ok, mx, rel = close(out[name], ref[name], tol)
        # also reported: the per-element rule with a fixed absolute floor
        floor = 1e-6 if w.dtype == "f32" else 1e-3
        _, _, erel = close_elementwise(out[name], ref[name], tol, floor)
        print(f"[err] {workload}.{name}: max abs {mx:.3e}, normwise rel {rel:.3e}, "
              f"max rel where |ref| > {floor / tol:.0e}: {erel:.3e}", flush=True)
        assert ok, f"{workload}.{name}: max abs err {mx:.3e}, normwise rel {rel:.3e} > tol {tol}"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("plan", PLANS)
@pytest.mark.parametrize("workload", list(FULL))
def test_full_size(workload, plan):
    print(f"\n[case] {workload} full {plan}", flush=True)
    w, r, raw, ref, out = run_plan(workload, FULL[workload], plan)
    check(workload, w, out, ref)


@pytest.mark.parametrize("plan", PLANS)
@pytest.mark.parametrize("workload", list(RAGGED))
def test_ragged(workload, plan):
    print(f"\n[case] {workload} ragged {RAGGED[workload]} {plan}", flush=True)
    w, r, raw, ref, out = run_plan(workload, RAGGED[workload], plan)
    check(workload, w, out, ref)


@pytest.mark.parametrize("workload", list(FULL))
def test_deterministic_rerun(workload):
    """Two executions of the fused plan give identical bytes (fixed reduction orders)."""
    print(f"\n[case] {workload} determinism", flush=True)
    w, r, raw, ref, out = run_plan(workload, FULL[workload], "fused")
    a = [t.clone() for t in r.outs]
    r.launch()
    torch.cuda.synchronize()
    for x, y in zip(a, r.outs):
        it = torch.int16 if x.element_size() == 2 else torch.int32
        assert torch.equal(x.view(it), y.view(it))
