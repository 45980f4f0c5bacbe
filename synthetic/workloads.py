"""Input recipes of the five synthetic workloads (shapes, dtypes, distributions, seeds).

Only the *inputs* are described here: names, shapes, storage dtype and the
distribution each tensor is drawn from.  The primitive graphs themselves are
built separately by the oracle and by the GPU path's Python binding.

Workloads (sizes are the defaults; every builder also accepts smaller or
ragged sizes for tests):

1. single-head attention, fp32: Q, K, V [128, 64] ~ N(0, 1)
2. transformer MLP block, fp16: X [4096, 768] ~ N(0,1); W1 [768, 3072] and
   W2 [3072, 768] ~ N(0, 0.02^2); gamma = 1 + N(0, 0.1^2); beta ~ N(0, 0.1^2)
3. spatial-reduction self-attention, fp16: X [128, 128, 64] ~ N(0,1);
   Wsr [8*8*64, 64] ~ N(0, 0.02^2); gamma, beta as in workload 2
4. conv + BN + Mish, fp16 NHWC: X [416, 416, 32] ~ N(0,1);
   W [3, 3, 32, 64] ~ N(0, 0.05^2); scale ~ U(0.5, 1.5); shift ~ N(0, 0.1^2)
5. ReLU linear attention, bf16: Q, K, V [16, 4096, 16] ~ N(0,1)
"""

from __future__ import annotations

from . import make_inputs

# (name, seed, shape, dtype, dist, a, b): a/b are mean/std for "normal" and
# low/high for "uniform".


def attention_specs(n=128, d=64, nk=None, dtype="f32"):
    nk = n if nk is None else nk
    return [
        ("Q", 1001, (n, d), dtype, "normal", 0.0, 1.0),
        ("K", 1002, (nk, d), dtype, "normal", 0.0, 1.0),
        ("V", 1003, (nk, d), dtype, "normal", 0.0, 1.0),
    ]


def mlp_specs(m=4096, d=768, h=3072, dtype="f16"):
    return [
        ("X", 2001, (m, d), dtype, "normal", 0.0, 1.0),
        ("W1", 2002, (d, h), dtype, "normal", 0.0, 0.02),
        ("W2", 2003, (h, d), dtype, "normal", 0.0, 0.02),
        ("gamma", 2004, (d,), dtype, "normal", 1.0, 0.1),
        ("beta", 2005, (d,), dtype, "normal", 0.0, 0.1),
    ]


def sra_specs(hh=128, ww=128, c=64, r=8, dtype="f16"):
    return [
        ("X", 3001, (hh, ww, c), dtype, "normal", 0.0, 1.0),
        ("Wsr", 3002, (r * r * c, c), dtype, "normal", 0.0, 0.02),
        ("gamma", 3003, (c,), dtype, "normal", 1.0, 0.1),
        ("beta", 3004, (c,), dtype, "normal", 0.0, 0.1),
    ]


def conv_specs(hh=416, ww=416, cin=32, cout=64, k=3, dtype="f16"):
    return [
        ("X", 4001, (hh, ww, cin), dtype, "normal", 0.0, 1.0),
        ("W", 4002, (k, k, cin, cout), dtype, "normal", 0.0, 0.05),
        ("scale", 4003, (cout,), dtype, "uniform", 0.5, 1.5),
        ("shift", 4004, (cout,), dtype, "normal", 0.0, 0.1),
    ]


def linattn_specs(heads=16, n=4096, d=16, dtype="bf16"):
    return [
        ("Q", 5001, (heads, n, d), dtype, "normal", 0.0, 1.0),
        ("K", 5002, (heads, n, d), dtype, "normal", 0.0, 1.0),
        ("V", 5003, (heads, n, d), dtype, "normal", 0.0, 1.0),
    ]


def instnorm_specs(hh=224, ww=224, c=32, dtype="f16"):
    # activations after a convolution: per-tensor offset and spread
    return [
        ("X", 6001, (hh, ww, c), dtype, "normal", 0.3, 1.2),
        ("gamma", 6002, (c,), dtype, "normal", 1.0, 0.1),
        ("beta", 6003, (c,), dtype, "normal", 0.0, 0.1),
    ]


SPEC_FNS = {
    "attention": attention_specs,
    "mlp": mlp_specs,
    "sra": sra_specs,
    "conv": conv_specs,
    "linattn": linattn_specs,
    "instnorm": instnorm_specs,
}

# Workload names in the order of the five configurations.
WORKLOADS = ("attention", "mlp", "sra", "conv", "linattn", "instnorm")

DEFAULT_DTYPE = {"attention": "f32", "mlp": "f16", "sra": "f16", "conv": "f16", "linattn": "bf16", "instnorm": "f16"}


def specs(workload: str, **shape):
    return SPEC_FNS[workload](**shape)


def inputs(workload: str, **shape):
    """``{name: storage_array}`` for one workload at the given sizes."""
    return make_inputs(specs(workload, **shape))
