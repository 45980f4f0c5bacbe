"""GPU tests of the GEMM family's direct-to-LDS operand staging.

Products whose operands are plain 16-bit tensors and whose tiles divide the
problem stage both operand tiles with direct global-to-LDS loads in swizzled
layouts (the MLP block's first product in the layered plan; asked for, the
second as eight waves over the whole contraction with three or five stages of
each operand).
The staging changes no arithmetic: every output element sums the same
products in the same k order, so each case must give the same bytes as the
register-staged kernel over the whole contraction (KORCH_GEMM_DMA=0 and
KORCH_GEMM_NO_KSPLIT=1) and match the float64 oracle within the dtype
tolerance.
Repeated executions, with and without a cache flush between them, must give
identical bytes (the waits before each barrier cover every load a tile
needs).
"""

import ctypes as C

import pytest

from paper_2406_09465_amd.warm import DMA8_CASES, DMA_CASES
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
    monkeypatch.delenv("KORCH_GEMM_DMA8", raising=False)
    monkeypatch.setenv("KORCH_GEMM_DMA_KSPLIT", "1")
    w, r, out, _, srcs = _run({}, raw)
    assert "global_load_lds_dwordx4" in srcs[2] and "kgrp" in srcs[2]
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
    # no intra-workgroup split of K in either run, so both sum each output's
    # products in one k order
    monkeypatch.setenv("KORCH_GEMM_NO_KSPLIT", "1")
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


@pytest.mark.parametrize("stages", ["3", "5"])
@pytest.mark.parametrize("sizes", [{}] + DMA8_CASES, ids=lambda s: "x".join(str(v) for v in s.values()) or "full")
def test_eight_wave_dma_matches_register_staging(sizes, stages, monkeypatch):
    """Second products on the eight-wave path (KORCH_GEMM_DMA8=1), 48 k-tiles
    and odd numbers of them (the loading groups of each operand take the
    k-tiles by residue mod 2, or mod 4 with five stages, so the last tiles fall
    to different groups): oracle parity, and the same bytes as register staging
    over the whole contraction."""
    print(f"\n[case] mlp {sizes} layered, eight waves, {stages} stages per operand", flush=True)
    raw, ref = reference("mlp", sizes)
    for var in ("KORCH_GEMM_DMA", "KORCH_GEMM_NO_KSPLIT", "KORCH_GEMM_DMA_2STAGE"):
        monkeypatch.delenv(var, raising=False)
    monkeypatch.setenv("KORCH_GEMM_DMA8", "1")
    monkeypatch.setenv("KORCH_GEMM_DMA_STAGES", stages)
    w, r, out, _, srcs = _run(sizes, raw)
    assert f"{stages} A stages and {stages} B stages" in srcs[2] and "kgrp" not in srcs[2]
    ok, mx, rel = close(out["out"], ref["out"], TOL[w.dtype])
    assert ok, f"mlp {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"
    monkeypatch.setenv("KORCH_GEMM_DMA", "0")
    monkeypatch.setenv("KORCH_GEMM_NO_KSPLIT", "1")
    monkeypatch.delenv("KORCH_GEMM_DMA8")
    monkeypatch.delenv("KORCH_GEMM_DMA_STAGES")
    _, r0, _, ndma0, _ = _run(sizes, raw)
    assert ndma0 == 0
    for a, b in zip(r.outs, r0.outs):
        assert a.dtype == b.dtype and torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("dma8", ["", "1"])
def test_dma_staging_repeats_bitwise(dma8, monkeypatch):
    """The full MLP block's layered plan (and with the second product on the
    eight-wave path), 100 back-to-back executions and 20 after a 512 MiB cache
    flush each (loads from HBM take longer than one k-tile's products):
    identical bytes every time."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd._abi import lib
    from paper_2406_09465_amd.runner import PlanRunner
    from synthetic import workloads as W
    for var in ("KORCH_GEMM_DMA", "KORCH_GEMM_DMA8", "KORCH_GEMM_NO_KSPLIT", "KORCH_GEMM_DMA_2STAGE", "KORCH_GEMM_DMA_STAGES"):
        monkeypatch.delenv(var, raising=False)
    if dma8:
        monkeypatch.setenv("KORCH_GEMM_DMA8", dma8)
    print(f"\n[case] mlp layered, direct-to-LDS staging, repeated, dma8={dma8}", flush=True)
    r = PlanRunner(graphs.build("mlp"), "layered")
    assert "global_load_lds_dwordx4" in r.plan.kernel_source(1)
    assert ("3 A stages and 3 B stages" in r.plan.kernel_source(2)) == bool(dma8)
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
