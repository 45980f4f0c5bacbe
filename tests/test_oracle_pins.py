"""Pins of the float64 oracle against closed forms, brute force and invariants.

Each test checks the oracle against something other than the oracle itself:
a textbook definition written out as loops, a closed form, an algebraic
identity, or a library routine on a special case.  The tests are chosen so a
plausible mistake (dropped term, wrong sign or index, transposed operand,
biased/unbiased variance, eps in the wrong place) fails at least one of them.
"""

import itertools
import math

import numpy as np
import pytest

from oracle import configs, primitives as P
from oracle.graph import Graph, run_unfused
from tests.helpers import inputs_f64


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# --------------------------------------------------------------------------
# Elementwise / reduce / layout / linear primitives against brute force
# --------------------------------------------------------------------------

def test_reduce_against_loops():
    x = rng(1).standard_normal((3, 4, 5))
    for axis in range(3):
        for op in ("reduce_sum", "reduce_mean", "reduce_max"):
            got = P.reduce(op, x, axis, keepdim=False)
            other = [d for d in range(3) if d != axis]
            ref = np.zeros([x.shape[d] for d in other])
            for idx in itertools.product(*[range(x.shape[d]) for d in other]):
                vals = []
                for k in range(x.shape[axis]):
                    full = list(idx)
                    full.insert(axis, k)
                    vals.append(x[tuple(full)])
                if op == "reduce_sum":
                    r = 0.0
                    for v in vals:
                        r += v
                elif op == "reduce_mean":
                    r = sum(vals) / len(vals)
                else:
                    r = max(vals)
                ref[idx] = r
            np.testing.assert_allclose(got, ref, rtol=1e-14, atol=1e-14)
            assert P.reduce(op, x, axis, keepdim=True).shape[axis] == 1


def test_transpose_reshape_against_loops():
    x = rng(2).standard_normal((2, 3, 4))
    perm = (2, 0, 1)
    t = P.transpose(x, perm)
    assert t.shape == (4, 2, 3)
    for i, j, k in itertools.product(range(4), range(2), range(3)):
        # output dim k' takes input dim perm[k']
        src = [0, 0, 0]
        src[perm[0]], src[perm[1]], src[perm[2]] = i, j, k
        assert t[i, j, k] == x[tuple(src)]
    r = P.reshape(x, (6, 4))
    flat = [x[a, b, c] for a in range(2) for b in range(3) for c in range(4)]
    assert list(r.ravel()) == flat


def test_slice_pad_concat_against_loops():
    x = rng(3).standard_normal((3, 4))
    s = P.slice_(x, (1, 0), (3, 3))
    assert s.shape == (2, 3) and all(s[i, j] == x[i + 1, j] for i in range(2) for j in range(3))
    p = P.pad(x, (1, 0), (0, 2), 7.5)
    assert p.shape == (4, 6)
    for i in range(4):
        for j in range(6):
            inside = 1 <= i < 4 and 0 <= j < 4
            assert p[i, j] == (x[i - 1, j] if inside else 7.5)
    c = P.concat([x, 2 * x], axis=1)
    assert c.shape == (3, 8) and np.all(c[:, :4] == x) and np.all(c[:, 4:] == 2 * x)


@pytest.mark.parametrize("shape_a,shape_b", [((3, 5), (5, 4)), ((1, 1), (1, 1)), ((7, 2), (2, 9)),
                                             ((2, 3, 4), (2, 4, 5)), ((2, 3, 4), (4, 5))])
def test_matmul_triple_loop(shape_a, shape_b):
    """T3: matrix product == triple loop (batched: per batch)."""
    a = rng(4).standard_normal(shape_a)
    b = rng(5).standard_normal(shape_b)
    got = P.matmul(a, b)
    A = a if a.ndim == 3 else a[None]
    B = b if b.ndim == 3 else np.broadcast_to(b, (A.shape[0],) + b.shape)
    ref = np.zeros((A.shape[0], A.shape[1], B.shape[2]))
    for bt in range(A.shape[0]):
        for i in range(A.shape[1]):
            for j in range(B.shape[2]):
                acc = 0.0
                for k in range(A.shape[2]):
                    acc += A[bt, i, k] * B[bt, k, j]
                ref[bt, i, j] = acc
    if a.ndim == 2:
        ref = ref[0]
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_conv_seven_loops():
    """T4: convolution (cross-correlation, zero padding) == direct 7-deep loop."""
    x = rng(6).standard_normal((5, 6, 3))
    w = rng(7).standard_normal((3, 3, 3, 4))
    for stride, pad in ((1, 1), (2, 1), (1, 0)):
        got = P.conv2d_nhwc(x, w, stride, pad)
        ho = (5 + 2 * pad - 3) // stride + 1
        wo = (6 + 2 * pad - 3) // stride + 1
        ref = np.zeros((ho, wo, 4))
        for y in range(ho):
            for xx in range(wo):
                for co in range(4):
                    acc = 0.0
                    for ky in range(3):
                        for kx in range(3):
                            for ci in range(3):
                                iy, ix = y * stride + ky - pad, xx * stride + kx - pad
                                if 0 <= iy < 5 and 0 <= ix < 6:
                                    acc += x[iy, ix, ci] * w[ky, kx, ci, co]
                    ref[y, xx, co] = acc
        np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_conv_delta_and_corner_taps():
    """T4: a centre delta copies channels; a corner tap shifts by (-1,-1) with a zero border."""
    x = rng(8).standard_normal((5, 6, 3))
    w = np.zeros((3, 3, 3, 3))
    w[1, 1] = np.eye(3)
    np.testing.assert_array_equal(P.conv2d_nhwc(x, w, 1, 1), x)
    w = np.zeros((3, 3, 3, 3))
    w[0, 0] = np.eye(3)
    out = P.conv2d_nhwc(x, w, 1, 1)
    assert np.all(out[0, :] == 0) and np.all(out[:, 0] == 0)
    np.testing.assert_array_equal(out[1:, 1:], x[:-1, :-1])


def test_gelu_tanh_identities():
    """T7: gelu(0)=0 and gelu(x) - gelu(-x) = x."""
    assert P.gelu_tanh(np.array([0.0]))[0] == 0.0
    x = np.linspace(-8, 8, 1001)
    np.testing.assert_allclose(P.gelu_tanh(x) - P.gelu_tanh(-x), x, rtol=0, atol=1e-15 * 8 + 1e-15)
    # known value of the tanh form at x = 1: 0.5 (1 + tanh(sqrt(2/pi) * 1.044715))
    assert abs(P.gelu_tanh(np.array([1.0]))[0] - 0.5 * (1 + math.tanh(math.sqrt(2 / math.pi) * 1.044715))) < 1e-15


def test_elementwise_scalar_is_right_operand():
    x = np.array([1.0, 2.0, 4.0])
    assert list(P.elementwise("sub", [x], 1.0)) == [0.0, 1.0, 3.0]
    assert list(P.elementwise("div", [x], 2.0)) == [0.5, 1.0, 2.0]
    assert list(P.elementwise("rsqrt", [x])) == [1.0, 1 / math.sqrt(2), 0.5]


# --------------------------------------------------------------------------
# Workload-level pins
# --------------------------------------------------------------------------

def test_softmax_rows_sum_to_one_and_match_eq1():
    """T1: softmax rows sum to 1; max-subtracted and plain exp/sum forms agree."""
    g = configs.attention(n=32, d=16)
    _, x = inputs_f64("attention", n=32, d=16)
    vals = run_unfused(g, x, keep_all=True)
    p = vals["P"]
    assert np.max(np.abs(p.sum(axis=1) - 1.0)) <= 1e-13
    s = x["Q"] @ x["K"].T / 4.0
    plain = np.exp(s) / np.exp(s).sum(axis=1, keepdims=True)
    np.testing.assert_allclose(p, plain, rtol=1e-14, atol=0)


def test_layernorm_fission_moments():
    """T2: before the affine step rows have mean 0 and variance v/(v+eps) with v the
    biased variance; equals (x - mean)/sqrt(var + eps)."""
    m, d = 64, 96
    g = configs.mlp(m=m, d=d, h=32)
    _, x = inputs_f64("mlp", m=m, d=d, h=32)
    vals = run_unfused(g, x, keep_all=True)
    xh = vals["Xh"]
    X = x["X"]
    assert np.max(np.abs(xh.mean(axis=1))) <= 1e-12 * np.max(np.abs(X))
    v = X.var(axis=1)  # biased
    np.testing.assert_allclose((xh ** 2).mean(axis=1), v / (v + 1e-5), rtol=1e-13)
    direct = (X - X.mean(axis=1, keepdims=True)) / np.sqrt(X.var(axis=1, keepdims=True) + 1e-5)
    np.testing.assert_allclose(xh, direct, rtol=1e-13, atol=1e-14)
    # affine step and residual
    y = direct * x["gamma"] + x["beta"]
    h = y @ x["W1"]
    out = h * 0.5 * (1 + np.tanh(math.sqrt(2 / math.pi) * (h + 0.044715 * h ** 3))) @ x["W2"] + X
    np.testing.assert_allclose(vals["out"], out, rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    """T5: V rows all equal c -> O = c; K rows all equal -> O = mean of V rows."""
    n, d = 16, 8
    g = configs.attention(n=n, d=d)
    r = rng(9)
    q, k, v = r.standard_normal((3, n, d))
    c = r.standard_normal(d)
    o = run_unfused(g, {"Q": q, "K": k, "V": np.tile(c, (n, 1))})["O"]
    np.testing.assert_allclose(o, np.tile(c, (n, 1)), rtol=1e-13, atol=1e-13)
    o = run_unfused(g, {"Q": q, "K": np.tile(k[0], (n, 1)), "V": v})["O"]
    np.testing.assert_allclose(o, np.tile(v.mean(axis=0), (n, 1)), rtol=1e-13, atol=1e-13)
    # log-sum-exp route
    s = q @ k.T / math.sqrt(d)
    lse = np.log(np.exp(s - s.max(1, keepdims=True)).sum(1, keepdims=True)) + s.max(1, keepdims=True)
    o = run_unfused(g, {"Q": q, "K": k, "V": v})["O"]
    np.testing.assert_allclose(o, np.exp(s - lse) @ v, rtol=1e-12, atol=1e-13)


def test_linear_attention_quadratic_form():
    """T6: factored form == O(N^2) form on sampled rows; V == c; zero query row -> 0."""
    h, n, d = 2, 64, 4
    g = configs.linattn(heads=h, n=n, d=d)
    _, x = inputs_f64("linattn", heads=h, n=n, d=d)
    x["Q"][1, 5, :] = -np.abs(x["Q"][1, 5, :])  # relu(q) == 0
    out = run_unfused(g, x)["out"]
    qr, kr, v = np.maximum(x["Q"], 0), np.maximum(x["K"], 0), x["V"]
    for hh in range(h):
        for t in (0, 7, 33, 63):
            w = np.array([qr[hh, t] @ kr[hh, s] for s in range(n)])
            ref = (w[:, None] * v[hh]).sum(0) / (w.sum() + 1e-6)
            np.testing.assert_allclose(out[hh, t], ref, rtol=1e-12, atol=1e-14)
    assert np.all(out[1, 5] == 0.0)
    c = 0.75
    out = run_unfused(g, {"Q": x["Q"], "K": x["K"], "V": np.full((h, n, d), c)})["out"]
    qs = np.einsum("htd,hd->ht", qr, kr.sum(1))
    np.testing.assert_allclose(out, c * (qs / (qs + 1e-6))[..., None] * np.ones(d), rtol=1e-12, atol=1e-15)


def test_mish_identity():
    """T8: x tanh(ln(1+e^x)) == x n/(n+2), n = e^x (e^x + 2); limits."""
    g = configs.conv(hh=4, ww=4, cin=2, cout=2)
    w = np.zeros((3, 3, 2, 2))
    w[1, 1] = np.eye(2)
    x = np.linspace(-20, 20, 32).reshape(4, 4, 2)
    out = run_unfused(g, {"X": x, "W": w, "scale": np.ones(2), "shift": np.zeros(2)})["Y"]
    ex = np.exp(x)
    n = ex * (ex + 2)
    # log(1 + e^x) loses about eps/e^x relative precision for x < 0 (the sum
    # rounds before the logarithm), so the bound follows that conditioning.
    bound = 4 * np.finfo(np.float64).eps * np.maximum(1.0, np.exp(-x))
    assert np.all(np.abs(out - x * n / (n + 2)) <= bound * np.abs(x * n / (n + 2)) + 1e-300)
    mid = np.abs(x) <= 8
    np.testing.assert_allclose(out[mid], (x * n / (n + 2))[mid], rtol=1e-12)
    assert abs(out.ravel()[-1] - 20.0) < 1e-12 and abs(out.ravel()[0]) < 1e-7
    z = run_unfused(g, {"X": np.zeros((4, 4, 2)), "W": w, "scale": np.ones(2), "shift": np.zeros(2)})["Y"]
    assert np.all(z == 0)


def test_bn_scale_shift_one_hot():
    """T13: BN as y = x*s + b per channel, checked before Mish via a one-hot input."""
    g = configs.conv(hh=3, ww=3, cin=2, cout=2)
    x = np.zeros((3, 3, 2))
    x[1, 1, 0] = 1.0
    w = np.zeros((3, 3, 2, 2))
    w[1, 1] = np.eye(2)
    s, b = np.array([2.0, 3.0]), np.array([0.5, -0.25])
    vals = run_unfused(g, {"X": x, "W": w, "scale": s, "shift": b}, keep_all=True)
    ref = np.broadcast_to(b, (3, 3, 2)).copy()
    ref[1, 1, 0] = 2.0 + 0.5
    np.testing.assert_array_equal(vals["B"], ref)


def test_patch_extract_bijection_and_inverse():
    """T9: the spatial-reduction patch extraction is a bijection with a known inverse."""
    hh, ww, c, r = 16, 8, 3, 4
    g = Graph()
    xi = g.input("X", (hh, ww, c))
    xr = g.op("reshape", [xi], shape=(hh // r, r, ww // r, r, c))
    xt = g.op("transpose", [xr], perm=(0, 2, 1, 3, 4))
    a = g.op("reshape", [xt], name="A", shape=((hh // r) * (ww // r), r * r * c))
    g.output(a)
    x = rng(10).standard_normal((hh, ww, c))
    A = run_unfused(g, {"X": x})["A"]
    assert sorted(A.ravel()) == sorted(x.ravel())
    # row p = (py, px) patch, column (ky, kx, ch)
    for py in range(hh // r):
        for px in range(ww // r):
            for ky in range(r):
                for kx in range(r):
                    for ch in range(c):
                        assert A[py * (ww // r) + px, (ky * r + kx) * c + ch] == x[py * r + ky, px * r + kx, ch]
    back = A.reshape(hh // r, ww // r, r, r, c).transpose(0, 2, 1, 3, 4).reshape(hh, ww, c)
    np.testing.assert_array_equal(back, x)


def test_output_magnitudes():
    """T14: output scales that justify a tolerance relative to max|ref|."""
    _, x = inputs_f64("linattn", heads=2, n=512)
    out = run_unfused(configs.linattn(heads=2, n=512), x)["out"]
    assert 1e-3 < np.median(np.abs(out)) < 1.0
    _, x = inputs_f64("mlp", m=64)
    out = run_unfused(configs.mlp(m=64), x)["out"]
    assert 0.7 < out.std() < 1.5


def test_workload_graph_sizes():
    """Primitive counts of the five workload graphs."""
    counts = {w: len(configs.build(w).primitives()) for w in configs.BUILDERS}
    assert counts == {"attention": 9, "mlp": 13, "sra": 23, "conv": 8, "linattn": 10, "instnorm": 13}


def _instnorm(x, gamma, beta, eps=1e-5):
    hh, ww, c = x.shape
    g = configs.instnorm(hh=hh, ww=ww, c=c, eps=eps)
    return run_unfused(g, {"X": x, "gamma": gamma, "beta": beta})["out"]


def test_instnorm_closed_forms():
    """InstanceNorm -> ReLU -> Pad (Candy pattern): a per-channel constant input
    normalizes to 0, so the interior is relu(beta); a +-1 input (half the pixels
    each) has mean 0 and biased variance 1, so it becomes
    relu(+-gamma / sqrt(1 + eps) + beta); the one-pixel border is zero."""
    rng = np.random.default_rng(3)
    hh, ww, c, eps = 6, 8, 5, 1e-5
    gamma = rng.normal(1.0, 0.3, c)
    beta = rng.normal(0.0, 0.5, c)
    x = np.broadcast_to(rng.normal(size=c), (hh, ww, c)).copy()
    out = _instnorm(x, gamma, beta, eps)
    assert out.shape == (hh + 2, ww + 2, c)
    assert np.all(out[0] == 0) and np.all(out[-1] == 0) and np.all(out[:, 0] == 0) and np.all(out[:, -1] == 0)
    # the mean of a constant carries a rounding residue of ~1e-16, which the
    # reciprocal standard deviation 1/sqrt(eps) ~ 316 amplifies
    assert np.allclose(out[1:-1, 1:-1], np.maximum(beta, 0.0), rtol=0, atol=1e-12)
    sign = np.where((np.arange(hh * ww) % 2) == 0, 1.0, -1.0).reshape(hh, ww, 1)
    x2 = np.broadcast_to(sign, (hh, ww, c)).copy()
    out2 = _instnorm(x2, gamma, beta, eps)
    expect = np.maximum(sign * gamma / np.sqrt(1.0 + eps) + beta, 0.0)
    assert np.allclose(out2[1:-1, 1:-1], expect, rtol=1e-14, atol=1e-14)


def test_instnorm_shift_invariance():
    """Adding a per-channel constant to the input changes nothing (the mean is
    subtracted); scaling by 2 changes only the eps term."""
    rng = np.random.default_rng(4)
    x = rng.normal(size=(7, 5, 6))
    gamma, beta = rng.normal(1, 0.2, 6), rng.normal(0, 0.2, 6)
    a = _instnorm(x, gamma, beta)
    b = _instnorm(x + rng.normal(size=6) * 3.0, gamma, beta)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    c = _instnorm(2.0 * x, gamma, beta, eps=4e-5)
    assert np.allclose(a, c, rtol=1e-12, atol=1e-12)


def _sra_direct(x, wsr, gamma, beta, r, eps=1e-5):
    """Spatial-reduction attention written out from its definition, with no
    primitive graph: patch matrix by loops in (ky, kx, c) order, the patch-merge
    product, biased LayerNorm with eps inside the square root, K = V = that
    result, scores scaled by 1/sqrt(c), SciPy's row softmax, then P V."""
    from scipy.special import softmax
    hh, ww, c = x.shape
    ph, pw = hh // r, ww // r
    a = np.zeros((ph * pw, r * r * c))
    for py in range(ph):
        for px in range(pw):
            for ky in range(r):
                for kx in range(r):
                    for ch in range(c):
                        a[py * pw + px, (ky * r + kx) * c + ch] = x[py * r + ky, px * r + kx, ch]
    kvp = a @ wsr
    kv = (kvp - kvp.mean(axis=1, keepdims=True)) / np.sqrt(kvp.var(axis=1, keepdims=True) + eps) * gamma + beta
    q = np.array([[x[i, j, ch] for ch in range(c)] for i in range(hh) for j in range(ww)])
    p = softmax(q @ kv.T / math.sqrt(c), axis=1)
    return p @ kv


@pytest.mark.parametrize("hh,ww,c,r", [(16, 16, 8, 2), (16, 24, 4, 4)])
def test_sra_graph_against_direct_formula(hh, ww, c, r):
    """The whole spatial-reduction attention graph (patch extraction, patch
    merge, fissioned LayerNorm, scaled scores, fissioned softmax, P KV) equals
    the attention formula computed directly, so a wrong permutation, scale,
    eps placement or K != V in the builder fails here."""
    g = rng(40 + r)
    x = g.standard_normal((hh, ww, c))
    wsr = g.standard_normal((r * r * c, c)) * 0.3
    gamma = 1.0 + 0.1 * g.standard_normal(c)
    beta = 0.1 * g.standard_normal(c)
    got = run_unfused(configs.sra(hh=hh, ww=ww, c=c, r=r),
                      {"X": x, "Wsr": wsr, "gamma": gamma, "beta": beta})["O"]
    ref = _sra_direct(x, wsr, gamma, beta, r)
    assert got.shape == (hh * ww, c)
    assert np.max(np.abs(got - ref)) <= 1e-13 * np.max(np.abs(ref))
    # the bound is tight enough to see even a 50 % change of eps
    wrong = _sra_direct(x, wsr, gamma, beta, r, eps=1e-5 * 1.5)
    assert np.max(np.abs(wrong - ref)) > 1e-9 * np.max(np.abs(ref))


@pytest.mark.parametrize("src,dst", [((3, 1), (2, 3, 4)), ((1,), (5,)), ((4,), (3, 4)), ((2, 1, 3), (2, 5, 3)),
                                     ((1, 1), (1, 1))])
def test_broadcast_against_loops(src, dst):
    """Broadcast replicates along size-1 and missing leading dimensions: output
    element x reads the input at x with the missing leading dimensions dropped
    and every size-1 dimension indexed at 0."""
    x = rng(50).standard_normal(src)
    got = P.broadcast(x, dst)
    assert got.shape == tuple(dst)
    lead = len(dst) - len(src)
    for idx in itertools.product(*[range(d) for d in dst]):
        tail = idx[lead:]
        sidx = tuple(0 if src[k] == 1 else tail[k] for k in range(len(src)))
        assert got[idx] == x[sidx]
    g = Graph()
    xi = g.input("X", src)
    b = g.op("broadcast", [xi], name="B", shape=dst)
    g.output(b)
    np.testing.assert_array_equal(run_unfused(g, {"X": x})["B"], got)
    # the result owns its memory (a later in-place change to it does not reach x)
    got.flat[0] += 1.0
    assert x.flat[0] != got.flat[0]
