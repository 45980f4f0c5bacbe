"""GPU parity of the GEMM family's folded LayerNorm against the float64 oracle.

A kernel holding the fissioned LayerNorm (mean, centred square, mean,
rsqrt, scale, affine) and the product it feeds stages the raw rows X,
multiplies X·diag(gamma) by W and evaluates LN(X)·W as
r·(X·diag(gamma)·W − mu·gammaᵀW) + betaᵀW, with mu, r from the row sums of X
and X² it accumulates from its own fragments and gammaᵀW, betaᵀW from its
right-operand fragments.  Plans with the GELU inside that kernel and with the
product as the kernel's output are compared with the oracle on every element,
and repeated executions must give identical bytes.
"""

import pytest

from paper_2406_09465_amd.warm import LN_FOLD_CASES, LN_FOLD_PLANS
from tests.helpers import TOL, close
from tests.test_gpu_parity import reference

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _runner(sizes, plan):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    w = graphs.build("mlp", **sizes)
    ks = [([w.ids[n] for n in p], [w.ids[n] for n in o]) for p, o in LN_FOLD_PLANS[plan]]
    r = PlanRunner(w, kernels=ks)
    assert "lnmu_" in r.plan.kernel_source(0)  # the folded LayerNorm
    return w, r


@pytest.mark.parametrize("plan", list(LN_FOLD_PLANS))
@pytest.mark.parametrize("sizes", LN_FOLD_CASES, ids=lambda s: "x".join(str(v) for v in s.values()) or "full")
def test_ln_fold_parity(sizes, plan):
    print(f"\n[case] mlp {sizes} folded LayerNorm, plan {plan}", flush=True)
    w, r = _runner(sizes, plan)
    raw, ref = reference("mlp", sizes)
    out = r.run(raw)
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    print(f"[err] max abs {mx:.3e}, normwise rel {rel:.3e}", flush=True)
    assert ok, f"mlp {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"


def test_ln_fold_repeats_bitwise():
    from synthetic import workloads as W
    print("\n[case] mlp folded LayerNorm, repeated", flush=True)
    _, r = _runner({}, "gelu")
    r.set_inputs(W.inputs("mlp"))
    r.launch()
    torch.cuda.synchronize()
    ref = [t.clone() for t in r.outs]
    for i in range(50):
        for t in r.outs:
            t.zero_()
        r.launch()
        torch.cuda.synchronize()
        assert all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(ref, r.outs)), f"execution {i}"
