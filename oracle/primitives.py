"""Float64 semantics of every primitive (Korch, Section 3, "Operator Fission").

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each function takes and returns ``numpy.float64`` arrays and materializes its
full output.  Nothing here fuses, reorders or blocks work beyond what the
definition states.

The four primitive categories (Section 3):
  * elementwise: O[x] = f(I1[x], ..., In[x]); operands of lower rank or with
    size-1 dimensions are broadcast implicitly, as in ONNX (Section 5.1 notes
    that broadcast is implicit in ONNX operators);
  * reduce: aggregate with an operator along one dimension k;
    broadcast: replicate along dimension k;
  * layout transformation: O[x] = I[L(x)] with L one-to-one (transpose,
    reshape, slice, pad, concat);
  * linear transformation: output linear in each input (matrix product,
    batched matrix product, convolution).
"""

from __future__ import annotations

import math

import numpy as np

# ----------------------------------------------------------------------------
# Elementwise primitives (Section 3, "Elementwise primitives")
# ----------------------------------------------------------------------------

_SQRT_2_OVER_PI = math.sqrt(2.0 / math.pi)


def gelu_tanh(x):
    """tanh-approximated GELU: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(_SQRT_2_OVER_PI * (x + 0.044715 * x * x * x)))


UNARY = {
    "neg": lambda x: -x,
    "exp": np.exp,
    "log": np.log,
    "tanh": np.tanh,
    "sqrt": np.sqrt,
    "rsqrt": lambda x: 1.0 / np.sqrt(x),
    "relu": lambda x: np.maximum(x, 0.0),
    "square": lambda x: x * x,
    "recip": lambda x: 1.0 / x,
    "gelu_tanh": gelu_tanh,
    "abs": np.abs,
    "identity": lambda x: x.copy(),
}

BINARY = {
    "add": np.add,
    "sub": np.subtract,
    "mul": np.multiply,
    "div": np.divide,
    "max": np.maximum,
    "min": np.minimum,
}


def elementwise(op: str, operands, scalar=None):
    """Apply elementwise primitive ``op``.

    Unary ops take one operand.  Binary ops take two operands, or one operand
    and ``scalar`` (the scalar is the right-hand operand: ``x op scalar``).
    Operands broadcast with NumPy's (ONNX's) right-aligned rule.
    """
    with np.errstate(over="ignore", divide="ignore", invalid="ignore"):
        if op in UNARY:
            (x,) = operands
            return np.asarray(UNARY[op](np.asarray(x, dtype=np.float64)), dtype=np.float64)
        if op in BINARY:
            if scalar is not None:
                (x,) = operands
                return BINARY[op](np.asarray(x, dtype=np.float64), np.float64(scalar))
            x, y = operands
            return BINARY[op](np.asarray(x, dtype=np.float64), np.asarray(y, dtype=np.float64))
    raise ValueError(f"not an elementwise primitive: {op}")


# ----------------------------------------------------------------------------
# Reduce and broadcast primitives (Section 3, "Reduce and broadcast primitives")
# ----------------------------------------------------------------------------


def reduce(op: str, x, axis: int, keepdim: bool):
    """Aggregate along dimension ``axis`` with sum, mean (sum / n) or max."""
    x = np.asarray(x, dtype=np.float64)
    if op == "reduce_sum":
        return np.sum(x, axis=axis, keepdims=keepdim)
    if op == "reduce_mean":
        return np.sum(x, axis=axis, keepdims=keepdim) / np.float64(x.shape[axis])
    if op == "reduce_max":
        return np.max(x, axis=axis, keepdims=keepdim)
    raise ValueError(f"not a reduce primitive: {op}")


def broadcast(x, shape):
    """Replicate ``x`` along its size-1 (or missing leading) dimensions."""
    return np.array(np.broadcast_to(np.asarray(x, dtype=np.float64), tuple(shape)))


# ----------------------------------------------------------------------------
# Layout transformation primitives (Section 3, "Layout transformation")
# ----------------------------------------------------------------------------


def transpose(x, perm):
    """O[x_0..x_{r-1}] = I[y] with y[perm[k]] = x[k]  (output dim k = input dim perm[k])."""
    return np.ascontiguousarray(np.transpose(np.asarray(x), tuple(perm)))


def reshape(x, shape):
    """Row-major reinterpretation with a new shape (same element count)."""
    return np.ascontiguousarray(np.asarray(x)).reshape(tuple(shape)).copy()


def slice_(x, begin, end):
    """O[x] = I[x + begin], for begin <= x + begin < end (unit step)."""
    idx = tuple(slice(int(b), int(e)) for b, e in zip(begin, end))
    return np.ascontiguousarray(np.asarray(x)[idx])


def pad(x, lo, hi, value):
    """Constant padding: ``lo[k]`` elements before and ``hi[k]`` after dimension k."""
    widths = [(int(a), int(b)) for a, b in zip(lo, hi)]
    return np.pad(np.asarray(x, dtype=np.float64), widths, mode="constant", constant_values=np.float64(value))


def concat(xs, axis):
    return np.concatenate([np.asarray(x, dtype=np.float64) for x in xs], axis=axis)


def fill(shape, value):
    """A constant tensor (no operands): the ones tensor of the transformation that
    writes a sum over an axis as a product (Section 3)."""
    return np.full(tuple(int(d) for d in shape), np.float64(value))


# ----------------------------------------------------------------------------
# Linear transformation primitives (Section 3, "Linear transformation")
# ----------------------------------------------------------------------------


def matmul(a, b):
    """Matrix product over the last two dimensions, batch dimensions broadcast."""
    return np.matmul(np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64))


def conv2d_nhwc(x, w, stride: int, pad_: int):
    """2-D cross-correlation, channels last, zero padding, no bias.

    x: [H, W, Cin] (or [N, H, W, Cin]); w: [KH, KW, Cin, Cout] (HWIO).
    out[y, x, co] = sum_{ky, kx, ci} xpad[y*stride + ky, x*stride + kx, ci] * w[ky, kx, ci, co]
    Computed as one matrix product per filter tap, summed over the taps.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    batched = x.ndim == 4
    if not batched:
        x = x[None]
    n, h, wd, cin = x.shape
    kh, kw, cin2, cout = w.shape
    assert cin == cin2, "channel mismatch"
    ho = (h + 2 * pad_ - kh) // stride + 1
    wo = (wd + 2 * pad_ - kw) // stride + 1
    xp = np.zeros((n, h + 2 * pad_, wd + 2 * pad_, cin), dtype=np.float64)
    xp[:, pad_:pad_ + h, pad_:pad_ + wd, :] = x
    out = np.zeros((n, ho, wo, cout), dtype=np.float64)
    for ky in range(kh):
        for kx in range(kw):
            patch = xp[:, ky:ky + stride * (ho - 1) + 1:stride, kx:kx + stride * (wo - 1) + 1:stride, :]
            out += np.matmul(patch, w[ky, kx])
    return out if batched else out[0]
