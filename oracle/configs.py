"""The oracle's own builders of the five workload primitive graphs.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each builder applies operator fission by hand (Korch, Section 3: a fission
rule rewrites an operator into an equivalent primitive graph) and returns an
oracle ``Graph``.  Broadcast is implicit in binary primitives, as in ONNX
(Section 5.1).  Every builder takes the sizes as keyword arguments so tests can
run small and ragged variants; the defaults are the full workload sizes.
"""

from __future__ import annotations

import math

from .graph import Graph


def _softmax_rows(g, s):
    """Softmax fission (Section 1, softmax equation; Section 3): exponentials,
    a row reduction, a broadcast and a division.  The row maximum is
    subtracted first; that shifts every exponent of a row by the same amount
    and leaves the quotient unchanged (a test checks both forms agree)."""
    m = g.op("reduce_max", [s], name="m", axis=-1, keepdim=True)
    z = g.op("sub", [s, m], name="Z")
    e = g.op("exp", [z], name="E")
    ssum = g.op("reduce_sum", [e], name="s", axis=-1, keepdim=True)
    return g.op("div", [e, ssum], name="P")


def _layernorm_rows(g, x, gamma, beta, eps, prefix=""):
    """LayerNorm fission over the last axis: mean, subtract, square, mean
    (biased variance), add eps, reciprocal square root, multiply, affine."""
    mu = g.op("reduce_mean", [x], name=prefix + "mu", axis=-1, keepdim=True)
    d = g.op("sub", [x, mu], name=prefix + "D")
    d2 = g.op("square", [d], name=prefix + "D2")
    var = g.op("reduce_mean", [d2], name=prefix + "var", axis=-1, keepdim=True)
    ve = g.op("add", [var], name=prefix + "ve", scalar=eps)
    r = g.op("rsqrt", [ve], name=prefix + "r")
    xh = g.op("mul", [d, r], name=prefix + "Xh")
    yg = g.op("mul", [xh, gamma], name=prefix + "Yg")
    return g.op("add", [yg, beta], name=prefix + "Y")


def attention(n=128, d=64, nk=None, dtype="f32"):
    """Single-head attention: S = Q K^T / sqrt(d), row softmax, O = P V."""
    nk = n if nk is None else nk
    g = Graph(dtype)
    q = g.input("Q", (n, d))
    k = g.input("K", (nk, d))
    v = g.input("V", (nk, d))
    kt = g.op("transpose", [k], name="KT", perm=(1, 0))
    s0 = g.op("matmul", [q, kt], name="S0")
    s = g.op("mul", [s0], name="S", scalar=1.0 / math.sqrt(d))
    p = _softmax_rows(g, s)
    o = g.op("matmul", [p, v], name="O")
    g.output(o)
    return g


def mlp(m=4096, d=768, h=3072, dtype="f16", eps=1e-5):
    """Pre-LN transformer MLP: out = X + GELU(LN(X) W1) W2 (no biases)."""
    g = Graph(dtype)
    x = g.input("X", (m, d))
    w1 = g.input("W1", (d, h))
    w2 = g.input("W2", (h, d))
    gamma = g.input("gamma", (d,))
    beta = g.input("beta", (d,))
    y = _layernorm_rows(g, x, gamma, beta, eps)
    h0 = g.op("matmul", [y, w1], name="H0")
    hg = g.op("gelu_tanh", [h0], name="Hg")
    z = g.op("matmul", [hg, w2], name="Zo")
    out = g.op("add", [z, x], name="out")
    g.output(out)
    return g


def sra(hh=128, ww=128, c=64, r=8, dtype="f16", eps=1e-5):
    """Efficient self-attention with spatial reduction ratio r, one head.

    Keys/values: non-overlapping r x r patches of the NHWC map, each flattened
    in (ky, kx, c) order, projected by Wsr, then LayerNorm; K = V = that
    result.  Queries are the map's pixels (no projection).  Scale 1/sqrt(c).
    """
    g = Graph(dtype)
    x = g.input("X", (hh, ww, c))
    wsr = g.input("Wsr", (r * r * c, c))
    gamma = g.input("gamma", (c,))
    beta = g.input("beta", (c,))
    xr = g.op("reshape", [x], name="Xr", shape=(hh // r, r, ww // r, r, c))
    xt = g.op("transpose", [xr], name="Xt", perm=(0, 2, 1, 3, 4))
    a = g.op("reshape", [xt], name="A", shape=((hh // r) * (ww // r), r * r * c))
    kvp = g.op("matmul", [a, wsr], name="KVp")
    kv = _layernorm_rows(g, kvp, gamma, beta, eps, prefix="ln_")
    q = g.op("reshape", [x], name="Qv", shape=(hh * ww, c))
    kt = g.op("transpose", [kv], name="KT", perm=(1, 0))
    s0 = g.op("matmul", [q, kt], name="S0")
    s = g.op("mul", [s0], name="S", scalar=1.0 / math.sqrt(c))
    p = _softmax_rows(g, s)
    o = g.op("matmul", [p, kv], name="O")
    g.output(o)
    return g


def conv(hh=416, ww=416, cin=32, cout=64, k=3, dtype="f16"):
    """3x3 stride-1 pad-1 NHWC convolution, inference BatchNorm as a
    per-channel scale and shift, then Mish = x * tanh(log(1 + exp(x)))."""
    g = Graph(dtype)
    x = g.input("X", (hh, ww, cin))
    w = g.input("W", (k, k, cin, cout))
    scale = g.input("scale", (cout,))
    shift = g.input("shift", (cout,))
    c = g.op("conv2d", [x, w], name="C", stride=1, pad=k // 2)
    b1 = g.op("mul", [c, scale], name="B1")
    b = g.op("add", [b1, shift], name="B")
    e = g.op("exp", [b], name="E")
    e1 = g.op("add", [e], name="E1", scalar=1.0)
    sp = g.op("log", [e1], name="SP")
    t = g.op("tanh", [sp], name="T")
    y = g.op("mul", [b, t], name="Y")
    g.output(y)
    return g


def linattn(heads=16, n=4096, d=16, dtype="bf16", eps=1e-6):
    """ReLU linear attention per head:
    out = relu(Q) (relu(K)^T V) / (relu(Q) sum_t relu(K)_t + eps)."""
    g = Graph(dtype)
    q = g.input("Q", (heads, n, d))
    k = g.input("K", (heads, n, d))
    v = g.input("V", (heads, n, d))
    qr = g.op("relu", [q], name="Qr")
    kr = g.op("relu", [k], name="Kr")
    krt = g.op("transpose", [kr], name="KrT", perm=(0, 2, 1))
    kvm = g.op("matmul", [krt, v], name="KVm")
    sk = g.op("reduce_sum", [kr], name="sK", axis=1, keepdim=True)
    num = g.op("matmul", [qr, kvm], name="num")
    skt = g.op("transpose", [sk], name="sKT", perm=(0, 2, 1))
    den0 = g.op("matmul", [qr, skt], name="den0")
    den = g.op("add", [den0], name="den", scalar=eps)
    out = g.op("div", [num, den], name="out")
    g.output(out)
    return g


def instnorm(hh=224, ww=224, c=32, dtype="f16", eps=1e-5):
    """Candy's InstanceNorm -> ReLU -> Pad pattern (Section 6 case study) in
    NHWC at batch 1: per-channel statistics over all pixels (mean, subtract,
    square, mean = biased variance, add eps, reciprocal square root), normalize,
    per-channel affine, ReLU, then one pixel of zero padding on each side of
    the two spatial axes for the next 3x3 convolution."""
    g = Graph(dtype)
    x = g.input("X", (hh, ww, c))
    gamma = g.input("gamma", (c,))
    beta = g.input("beta", (c,))
    xp = g.op("reshape", [x], name="Xp", shape=(hh * ww, c))
    mu = g.op("reduce_mean", [xp], name="mu", axis=0, keepdim=True)
    d = g.op("sub", [xp, mu], name="D")
    d2 = g.op("square", [d], name="D2")
    var = g.op("reduce_mean", [d2], name="var", axis=0, keepdim=True)
    ve = g.op("add", [var], name="ve", scalar=eps)
    r = g.op("rsqrt", [ve], name="r")
    xh = g.op("mul", [d, r], name="Xh")
    yg = g.op("mul", [xh, gamma], name="Yg")
    y = g.op("add", [yg, beta], name="Y")
    rl = g.op("relu", [y], name="R")
    ri = g.op("reshape", [rl], name="Ri", shape=(hh, ww, c))
    out = g.op("pad", [ri], name="out", lo=(1, 1, 0), hi=(1, 1, 0), value=0.0)
    g.output(out)
    return g


BUILDERS = {"attention": attention, "mlp": mlp, "sra": sra, "conv": conv, "linattn": linattn, "instnorm": instnorm}


def build(workload: str, **shape):
    return BUILDERS[workload](**shape)
