"""GPU parity of the attention family's two kernels against the float64 oracle.

With few query rows the keys are split over the four waves of a workgroup
(one workgroup per 16 query rows, row statistics and partial P.V products
combined through LDS); otherwise each wave takes 16 query rows over all keys.
Cases: fp32 single-head attention (50 queries with 50 keys padded to 64, and
128 x 64), and fp16 spatial-reduction attention with 128 and 112 keys (the
latter padded to 128), each with the key split and without it
(KORCH_ATTN_NO_KEY_SPLIT=1).
"""

import pytest

from paper_2406_09465_amd.warm import ATTN_CASES
from tests.helpers import TOL, close
from tests.test_gpu_parity import reference

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("no_split", ["", "1"])
@pytest.mark.parametrize("case", ATTN_CASES, ids=lambda c: c[0] + "-" + "x".join(str(v) for v in c[1].values()))
def test_attention_kernels(case, no_split, monkeypatch):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    workload, sizes = case
    if no_split:
        monkeypatch.setenv("KORCH_ATTN_NO_KEY_SPLIT", no_split)
    else:
        monkeypatch.delenv("KORCH_ATTN_NO_KEY_SPLIT", raising=False)
    print(f"\n[case] {workload} {sizes} no_split={no_split}", flush=True)
    w = graphs.build(workload, **sizes)
    raw, ref = reference(workload, sizes)
    out = PlanRunner(w, "fused").run(raw)
    for name in w.output_names:
        ok, mx, rel = close(out[name], ref[name], TOL[w.dtype])
        assert ok, f"{workload} {sizes}: max abs err {mx:.3e}, normwise rel {rel:.3e}"
