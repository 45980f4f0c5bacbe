"""GPU tests of the GEMM family's direct-to-LDS operand staging.

Products whose operands are plain 16-bit tensors and whose tiles divide the
problem stage both operand tiles with direct global-to-LDS loads in swizzled
layouts (the MLP block's first product in the layered plan).  The staging
changes no arithmetic: the same MFMAs run in the same order on the same
values, so each case must give the same bytes as the register-staged kernel
(KORCH_GEMM_DMA=0) and match the float64 oracle within the dtype tolerance.
Repeated executions, with and without a cache flush between them, must give
identical bytes (the waits before each barrier cover every load a tile
needs).
"""

import ctypes as C

import pytest

from paper_2406_09465_amd.warm import DMA_CASES
from tests.helpers import TOL, close
from tests.test_gpu_parity import reference

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(sizes, raw):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    w = graphs.build("mlp", **sizes)
    r = PlanRunner(w, "layered")
    srcs = [r.plan.kernel_source(i) for i in range(r.plan.num_kernels())]
    return w, r, r.run(raw), sum("global_load_lds_dwordx4" in s for s in srcs), srcs


def test_dma_staging_k_split_matches_register_staging(monkeypatch):
    """The MLP block's second product (an intra-workgroup split of K) with
    direct-to-LDS staging asked for (KORCH_GEMM_DMA_KSPLIT=1): oracle parity
    and the same bytes as register staging."""
    print("\n[case] mlp layered, k-split product with direct-to-LDS staging", flush=True)
    raw, ref = reference("mlp", {})
    monkeypatch.delenv("KORCH_GEMM_DMA", raising=False)
    monkeypatch.setenv("KORCH_GEMM_DMA_KSPLIT", "1")
    w, r, out, _, srcs = _run({}, raw)
    assert "global_load_lds_dwordx4" in srcs[2]
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    assert ok, f"max abs err {mx:.3e}, normwise rel {rel:.3e}"
    monkeypatch.delenv("KORCH_GEMM_DMA_KSPLIT")
    _, r0, _, _, srcs0 = _run({}, raw)
    assert "global_load_lds_dwordx4" not in srcs0[2]
    for a, b in zip(r.outs, r0.outs):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("stages", ["", "2"])
@pytest.mark.parametrize("sizes", [{}] + DMA_CASES, ids=lambda s: "x".join(str(v) for v in s.values()) or "full")
def test_dma_staging_matches_register_staging(sizes, stages, monkeypatch):
    if stages and sizes:
        pytest.skip("two stages forced only on the full block")
    print(f"\n[case] mlp {sizes} layered, direct-to-LDS staging, stages={stages or 'default'}", flush=True)
    raw, ref = reference("mlp", sizes)
    monkeypatch.delenv("KORCH_GEMM_DMA", raising=False)
    if stages:
        monkeypatch.setenv("KORCH_GEMM_DMA_2STAGE", "1")
    else:
        monkeypatch.delenv("KORCH_GEMM_DMA_2STAGE", raising=False)
    w, r, out, ndma, srcs = _run(sizes, raw)
    assert ndma >= 1
    want = "2 B stages" if stages else None
    if want:
        assert any(want in s for s in srcs)
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    assert ok, f"mlp {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"
    monkeypatch.setenv("KORCH_GEMM_DMA", "0")
    monkeypatch.delenv("KORCH_GEMM_DMA_2STAGE", raising=False)
    _, r0, _, ndma0, _ = _run(sizes, raw)
    assert ndma0 == 0
    for a, b in zip(r.outs, r0.outs):
        assert a.dtype == b.dtype and torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_dma_staging_repeats_bitwise(monkeypatch):
    """The full MLP block's layered plan, 100 back-to-back executions and 20
    after a 512 MiB cache flush each (loads from HBM take longer than one
    k-tile's products): identical bytes every time."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd._abi import lib
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W
    monkeypatch.delenv("KORCH_GEMM_DMA", raising=False)
    monkeypatch.delenv("KORCH_GEMM_DMA_2STAGE", raising=False)
    print("\n[case] mlp layered, direct-to-LDS staging, repeated", flush=True)
    r = PlanRunner(graphs.build("mlp"), "layered")
    assert any("global_load_lds_dwordx4" in r.plan.kernel_source(i) for i in range(r.plan.num_kernels()))
    r.set_inputs(W.inputs("mlp"))
    r.launch()
    torch.cuda.synchronize()
    ref = [t.clone() for t in r.outs]
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    for i in range(120):
        for t in r.outs:
            t.zero_()
        if i >= 100:
            assert lib.korch_flush_caches(C.c_void_p(flush.data_ptr()), C.c_size_t(flush.numel()), 0,
                                          C.c_void_p(s.cuda_stream)) == 0
        r.launch()
        torch.cuda.synchronize()
        assert all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(ref, r.outs)), f"execution {i}"
