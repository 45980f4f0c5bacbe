"""GPU parity of the conv family's two kernels against the float64 oracle.

The direct kernel (input halo tile in LDS, weights in registers) serves
half-precision stride-1 convolutions whose weights fit its register budget; the
implicit-GEMM kernel serves the rest and is forced here with
KORCH_CONV_DIRECT=0.  The shapes cover padded input channels (8, and 48 as
two 32-channel chunks), three output fragments per wave (48 channels), output
channels that are not a multiple of 16 (24), a 5x5 filter, narrow images
(16-pixel-wide tiles), ragged tiles on both axes, and 128 output channels
(implicit GEMM only).
"""

import pytest

from paper_2406_09465_amd.warm import CONV_CASES as CASES
from tests.helpers import TOL, close
from tests.test_gpu_parity import reference

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(sizes, plan):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    w = graphs.build("conv", **sizes)
    raw, ref = reference("conv", sizes)
    r = PlanRunner(w, plan)
    return w, r.run(raw), ref


@pytest.mark.parametrize("direct", ["1", "0"])
@pytest.mark.parametrize("plan", ["fused", "layered"])
@pytest.mark.parametrize("sizes", CASES, ids=lambda s: "x".join(str(v) for v in s.values()))
def test_conv_kernels(sizes, plan, direct, monkeypatch):
    monkeypatch.setenv("KORCH_CONV_DIRECT", direct)
    print(f"\n[case] conv {sizes} {plan} direct={direct}", flush=True)
    w, out, ref = _run(sizes, plan)
    ok, mx, rel = close(out["Y"], ref["Y"], TOL[w.dtype])
    assert ok, f"conv {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"


def test_implicit_gemm_full_size(monkeypatch):
    """The implicit-GEMM kernel on the 416 x 416 x 32 -> 64 workload."""
    monkeypatch.setenv("KORCH_CONV_DIRECT", "0")
    print("\n[case] conv full implicit GEMM", flush=True)
    w, out, ref = _run({}, "fused")
    ok, mx, rel = close(out["Y"], ref["Y"], TOL[w.dtype])
    assert ok, f"conv full: max abs err {mx:.3e}, normwise rel {rel:.3e}"
