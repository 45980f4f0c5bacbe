"""GPU parity of the GEMM family's intra-workgroup split of K against the
float64 oracle.

GEMM2 of an MLP block whose tiles leave one workgroup per compute unit and
whose contraction is long runs as two groups of four waves over the two halves
of the k-tiles; the shapes cover an odd number of k-tiles (the second group
runs one tile fewer) with ragged rows, and an even number.  Each case also runs
with the split switched off (KORCH_GEMM_NO_KSPLIT=1).
"""

import pytest

from paper_2406_09465_amd.warm import GEMM_CASES
from tests.helpers import TOL, close
from tests.test_gpu_parity import reference

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("no_split", ["", "1"])
@pytest.mark.parametrize("plan", ["layered", "fused"])
@pytest.mark.parametrize("sizes", GEMM_CASES, ids=lambda s: "x".join(str(v) for v in s.values()))
def test_gemm_k_split(sizes, plan, no_split, monkeypatch):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    monkeypatch.delenv("KORCH_GEMM_NO_KSPLIT", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA8", raising=False)
    if no_split:
        monkeypatch.setenv("KORCH_GEMM_NO_KSPLIT", no_split)
    print(f"\n[case] mlp {sizes} {plan} no_split={no_split}", flush=True)
    w = graphs.build("mlp", **sizes)
    raw, ref = reference("mlp", sizes)
    out = PlanRunner(w, plan).run(raw)
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    assert ok, f"mlp {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"


@pytest.mark.parametrize("plan", ["layered", "fused"])
@pytest.mark.parametrize("case", ["wide", "big"])
def test_gemm_wide_tiles(plan, case):
    """128 x 192 tiles with k-tiles of 32, and 256 x 192 tiles of eight waves
    with k-tiles of 64 (ragged rows and contraction in both)."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    from paper_2406_09465_amd.warm import BIG_TILE_CASE, WIDE_TILE_CASE
    sizes = WIDE_TILE_CASE if case == "wide" else BIG_TILE_CASE
    print(f"\n[case] mlp {sizes} {plan} {case} tiles", flush=True)
    w = graphs.build("mlp", **sizes)
    raw, ref = reference("mlp", sizes)
    out = PlanRunner(w, plan).run(raw)
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    assert ok, f"mlp {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"
