"""GPU tests of the column-reduction family's one-pass moments.

An InstanceNorm after the split-moments transformation (its variance squares
m - X, a node of its own) runs as two kernels: the column moments (the mean
and the reciprocal deviation in one pass over X: Welford's update per thread,
Chan's pairwise merge across lanes, waves and splits in a fixed order) and
the rest (X - m recomputed, normalization, ReLU, pad).  The transformation
changes no value, so every case must match the float64 oracle of the original
graph: the output with the standard tolerance rule, the mean and the
reciprocal deviation (exported as extra outputs) per element within a few
fp16 units.  Zero-variance channels, a mean far from zero and repeated
executions (identical bytes) are covered too.
"""

import numpy as np
import pytest

from oracle import configs as OC
from oracle.graph import run_unfused
from paper_2406_09465_amd.warm import MOMENTS_CASES
from synthetic import round_to_storage, storage_to_f64
from synthetic.edge import edge_inputs
from tests.helpers import TOL, close, close_elementwise, inputs_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _runner(sizes):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    w2, n = graphs.rewritten(graphs.build("instnorm", extra_outputs=("mu", "r"), **sizes))
    assert n >= 1
    ks = graphs.moments_plan(w2)
    assert ks is not None and len(ks) == 2
    r = PlanRunner(w2, kernels=ks)
    src = r.plan.kernel_source(0)
    assert "korch_k0_colreduce" in src and "cn_ += 1.0f" in src  # the one-pass moments kernel
    return r


def _reference(sizes, raw):
    x = {k: storage_to_f64(v, "f16") for k, v in raw.items()}
    return run_unfused(OC.build("instnorm", **sizes), x, keep_all=True)


def _check(sizes, raw, what):
    ref = _reference(sizes, raw)
    out = _runner(sizes).run(raw)
    ok, mx, rel = close(out["out"], ref["out"], TOL["f16"])
    assert ok, f"{what} out: max abs err {mx:.3e}, normwise rel {rel:.3e}"
    # the mean (fp16 storage) and the reciprocal deviation per element: a few
    # fp16 units relative, with an absolute floor for means near zero
    ok, mx, rel = close_elementwise(out["mu"], ref["mu"], 2e-3, 2e-5)
    assert ok, f"{what} mu: max abs {mx:.3e}, max rel {rel:.3e}"
    ok, mx, rel = close_elementwise(out["r"], ref["r"], 2e-3, 0.0)
    assert ok, f"{what} r: max abs {mx:.3e}, max rel {rel:.3e}"
    return out, ref


@pytest.mark.parametrize("sizes", MOMENTS_CASES, ids=lambda s: "x".join(str(v) for v in s.values()) or "full")
def test_moments_plan_matches_oracle(sizes):
    print(f"\n[case] instnorm {sizes} moments plan", flush=True)
    raw, _ = inputs_f64("instnorm", **sizes)
    _check(sizes, raw, f"instnorm {sizes}")


def test_moments_zero_variance_channels():
    """Constant channels (0.3, -1.5, 0, 2.25): Welford's M2 stays exactly 0 and
    the merges add nothing, so the normalized values are exactly 0 and the
    output is ReLU(beta) in the interior, 0 on the pad border."""
    print("\n[case] instnorm moments plan, zero-variance channels", flush=True)
    raw = edge_inputs("instnorm")
    out, ref = _check({}, raw, "edge")
    x = {k: storage_to_f64(v, "f16") for k, v in raw.items()}
    beta = np.maximum(x["beta"][:4], 0.0)
    assert np.max(np.abs(out["out"][1:-1, 1:-1, :4] - beta)) <= 1e-3
    assert np.all(out["out"][0] == 0) and np.all(out["out"][:, 0] == 0)


def test_moments_mean_far_from_zero():
    """X + 100 (stored in fp16, spacing 1/16 there): the one-pass moments keep
    the variance of the centred values (no E[X^2] - E[X]^2 cancellation)."""
    print("\n[case] instnorm moments plan, X + 100", flush=True)
    raw, _ = inputs_f64("instnorm")
    raw = dict(raw)
    raw["X"] = round_to_storage((storage_to_f64(raw["X"], "f16") + 100.0).astype(np.float32), "f16")
    _check({}, raw, "offset")


def test_moments_repeats_bitwise():
    """Twenty executions of the full-size plan give identical bytes (fixed
    merge order; the last workgroup of the split resets its counters)."""
    print("\n[case] instnorm moments plan, repeated", flush=True)
    raw, _ = inputs_f64("instnorm")
    r = _runner({})
    r.set_inputs(raw)
    r.launch()
    torch.cuda.synchronize()
    first = [t.clone() for t in r.outs]
    for i in range(20):
        for t in r.outs:
            t.zero_()
        r.launch()
        torch.cuda.synchronize()
        assert all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(first, r.outs)), f"execution {i}"
