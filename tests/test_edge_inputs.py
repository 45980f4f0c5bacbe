"""The edge-case inputs produce the degenerate cases they are meant to, and
the oracle handles those cases as the definitions say (CPU only).

Each check compares the oracle with a closed form that holds on the edge
input: exact zeros of ReLU linear attention, LayerNorm / InstanceNorm of a
zero-variance row or channel reducing to the affine shift, Mish equal to its
argument above 20 and to 0 far below, and softmax rows that still sum to 1
when the scores spread over tens.
"""

import numpy as np

from oracle import configs as OC
from oracle.graph import run_unfused
from synthetic import storage_to_f64
from synthetic import workloads as W
from synthetic.edge import CASES, edge_inputs

SMALL = {
    "attention": dict(n=50, d=24),
    "mlp": dict(m=40, d=96, h=64),
    "sra": dict(hh=32, ww=16, c=16, r=8),
    "conv": dict(hh=9, ww=7, cin=8, cout=16),
    "linattn": dict(heads=3, n=50, d=16),
    "instnorm": dict(hh=6, ww=5, c=8),
}


def run(workload, keep_all=True):
    sz = SMALL[workload]
    raw = edge_inputs(workload, **sz)
    dt = W.DEFAULT_DTYPE[workload]
    x = {k: storage_to_f64(v, dt) for k, v in raw.items()}
    return x, run_unfused(OC.build(workload, **sz), x, keep_all=keep_all)


def test_every_workload_has_an_edge_case():
    assert set(CASES) == set(W.SPEC_FNS)
    for w in CASES:
        raw = edge_inputs(w, **SMALL[w])
        reg = W.inputs(w, **SMALL[w])
        assert raw.keys() == reg.keys()
        assert all(raw[k].shape == reg[k].shape and raw[k].dtype == reg[k].dtype for k in raw)


def test_linattn_zero_rows_are_exactly_zero():
    x, v = run("linattn")
    out = v["out"]
    assert np.all(out[:, ::7, :] == 0.0)
    assert np.all(out[2] == 0.0)
    assert np.all(v["sK"][2] == 0.0) and np.all(v["KVm"][2] == 0.0)
    assert np.count_nonzero(out[0, 1]) > 0


def test_mlp_flat_rows_normalize_to_beta():
    x, v = run("mlp")
    y = v["Y"]
    beta = x["beta"]
    for i in range(17):
        assert v["var"][i, 0] == 0.0
        np.testing.assert_allclose(y[i], beta, rtol=0, atol=1e-12)
    # the alternating row has mean 0 and biased variance exactly 1
    assert v["mu"][17, 0] == 0.0 and v["var"][17, 0] == 1.0


def test_instnorm_flat_channels_become_relu_beta():
    x, v = run("instnorm")
    out = v["out"]
    for ch in range(4):
        assert v["var"][0, ch] < 1e-28
        np.testing.assert_allclose(out[1:-1, 1:-1, ch], max(x["beta"][ch], 0.0), rtol=0, atol=1e-9)


def test_conv_wide_shift_covers_both_mish_limits():
    x, v = run("conv")
    b, y = v["B"], v["Y"]
    assert b.min() < -100 and b.max() > 100
    big = b > 20
    np.testing.assert_allclose(y[big], b[big], rtol=1e-15)
    tiny = b < -100
    assert np.all(np.abs(y[tiny]) < 1e-40) and np.all(y[tiny] <= 0)


def test_wide_scores_still_give_stochastic_rows():
    for w in ("attention", "sra"):
        x, v = run(w)
        s, p = v["S"], v["P"]
        assert s.max() - s.min() > 40
        np.testing.assert_allclose(p.sum(axis=-1), 1.0, rtol=0, atol=1e-13)
        assert np.mean(p < 1e-6) > 0.3
