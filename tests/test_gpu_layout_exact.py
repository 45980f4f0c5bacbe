"""GPU parity of layout primitives, bit for bit.

A layout primitive moves values without arithmetic: O[x] = I[L(x)] with L one
to one (Korch, Section 3, layout transformation primitives).  So every layout
kernel's output must equal, bit for bit, the oracle's layout function applied
to the very bits that kernel read: no tolerance applies.

Two kinds of cases:
  * in place: a workload's unfused plan (one kernel per primitive) with the
    layout node's operand and result marked as extra graph outputs, so the
    kernel that runs is the unfused plan's own layout kernel and both of its
    tensors can be read back (full workload size and a ragged size);
  * stand-alone: one layout primitive on seeded inputs that carry signed
    zeros, subnormals, infinities, the largest finite value and a quiet NaN,
    at the shapes of the slices and concatenations the product-merging
    transformation creates and at ragged shapes.
"""

import numpy as np
import pytest

from oracle import primitives as P
from synthetic import round_to_storage, storage_to_f64
from synthetic import workloads as W
from paper_2406_09465_amd.warm import LAYOUT_IN_PLACE, LAYOUT_SIZES, LAYOUT_STANDALONE

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BITS = {"f32": np.uint32, "f16": np.uint16, "bf16": np.uint16}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def device_bits(t):
    """Raw storage bits of a device tensor."""
    it = torch.int32 if t.element_size() == 4 else torch.int16
    return t.detach().contiguous().view(it).cpu().numpy().view(BITS["f32" if t.element_size() == 4 else "f16"])


def storage_bits(arr, dtype):
    """Raw bits of a storage array (float32 / float16 / uint16 bf16 bits)."""
    a = np.ascontiguousarray(arr)
    return a.view(BITS[dtype]) if dtype != "bf16" else a.astype(np.uint16)


def to_storage_bits(x64, dtype):
    """Bits of float64 values that are exactly representable in ``dtype``
    (every layout result here is): the rounding does not change them."""
    return storage_bits(round_to_storage(np.asarray(x64, dtype=np.float32), dtype), dtype)


def bits_to_f64(bits, dtype):
    if dtype == "bf16":
        return storage_to_f64(bits.astype(np.uint16), "bf16")
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    return bits.view(np.float32).astype(np.float64)


def assert_bits_equal(got, want, what):
    assert got.shape == want.shape, (what, got.shape, want.shape)
    bad = np.flatnonzero(got.ravel() != want.ravel())
    assert bad.size == 0, f"{what}: {bad.size} elements differ, first at {bad[0]}: " \
                          f"{int(got.ravel()[bad[0]]):#x} != {int(want.ravel()[bad[0]]):#x}"


# workload -> [(layout node, its operand: a graph input or a computed node)],
# and the sizes; the stand-alone cases: (op, dtype, input shapes, attributes)
IN_PLACE = {w: cases for w, cases in LAYOUT_IN_PLACE.items()}
IN_PLACE_CASES = [(w, sz) for w in LAYOUT_IN_PLACE for sz in LAYOUT_SIZES[w]]
STANDALONE = LAYOUT_STANDALONE
PERM = {("attention", "KT"): (1, 0), ("sra", "KT"): (1, 0), ("linattn", "KrT"): (0, 2, 1), ("linattn", "sKT"): (0, 2, 1)}


def _sra_patches(x, sizes):
    hh, ww, c = x.shape
    r = sizes.get("r", 8)
    return P.transpose(P.reshape(x, (hh // r, r, ww // r, r, c)), (0, 2, 1, 3, 4))


def _instnorm_pad(rows, sizes):
    hh, ww, c = sizes.get("hh", 224), sizes.get("ww", 224), sizes.get("c", 32)
    return P.pad(P.reshape(rows, (hh, ww, c)), (1, 1, 0), (1, 1, 0), 0.0)


@pytest.mark.parametrize("workload,sizes", IN_PLACE_CASES,
                         ids=[f"{w}-{'full' if not s else 'ragged'}" for w, s in IN_PLACE_CASES])
def test_unfused_layout_kernels_bit_exact(workload, sizes):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    print(f"\n[case] layout in place {workload} {sizes}", flush=True)
    cases = IN_PLACE[workload]
    inputs = {s[0] for s in W.specs(workload, **sizes)}
    extra = [n for node, operand in cases for n in (node, operand) if n not in inputs]
    w = graphs.build(workload, extra_outputs=extra, **sizes)
    raw = W.inputs(workload, **sizes)
    r = PlanRunner(w, "unfused")
    r.set_inputs(raw)
    r.launch()
    torch.cuda.synchronize()
    got = {name: device_bits(t) for name, t in zip(w.output_names, r.outs)}
    dt = w.dtype
    for node, operand in cases:
        src = storage_bits(raw[operand], dt) if operand in inputs else got[operand]
        x = bits_to_f64(src, dt)
        if workload == "sra" and node == "Xt":
            want = _sra_patches(x, sizes)
        elif workload == "instnorm":
            want = _instnorm_pad(x, sizes)
        else:
            want = P.transpose(x, PERM[(workload, node)])
        assert_bits_equal(got[node], to_storage_bits(want, dt).reshape(got[node].shape), f"{workload}.{node}")
    if workload == "linattn":
        # ReLU of a representable value is representable: Kr equals relu(K) exactly
        k = storage_to_f64(raw["K"], dt)
        np.testing.assert_array_equal(bits_to_f64(got["Kr"], dt).reshape(k.shape), np.maximum(k, 0.0))


@pytest.mark.parametrize("plan", ["fused", "layered"])
def test_instnorm_pad_border_is_exactly_zero(plan):
    """The fused normalize-ReLU-pad kernel writes the one-pixel border as +0.0."""
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    print(f"\n[case] instnorm border {plan}", flush=True)
    w = graphs.build("instnorm")
    r = PlanRunner(w, plan)
    r.set_inputs(W.inputs("instnorm"))
    r.launch()
    torch.cuda.synchronize()
    out = device_bits(r.outs[0])
    assert out.shape == (226, 226, 32)
    for border in (out[0], out[-1], out[:, 0], out[:, -1]):
        assert np.all(border == 0)
    assert np.count_nonzero(out[1:-1, 1:-1]) > 0


# Special values placed at the start of every stand-alone input (bits per dtype):
# +0, -0, smallest and largest subnormal, largest finite, +inf, -inf, quiet NaN.
SPECIAL = {
    "f32": [0x00000000, 0x80000000, 0x00000001, 0x007FFFFF, 0x7F7FFFFF, 0x7F800000, 0xFF800000, 0x7FC00000],
    "f16": [0x0000, 0x8000, 0x0001, 0x03FF, 0x7BFF, 0x7C00, 0xFC00, 0x7E00],
    "bf16": [0x0000, 0x8000, 0x0001, 0x007F, 0x7F7F, 0x7F80, 0xFF80, 0x7FC0],
}


def probe_input(seed, shape, dtype):
    """Seeded N(0,1) storage values with the special bit patterns in front."""
    from synthetic import make_tensor
    a = make_tensor(seed, shape, dtype, "normal", 0.0, 1.0)
    bits = storage_bits(a, dtype).copy().ravel()
    sp = np.array(SPECIAL[dtype], dtype=bits.dtype)
    bits[:min(sp.size, bits.size)] = sp[:bits.size]
    return bits.reshape(shape)


def _raw_from_bits(bits, dtype):
    if dtype == "bf16":
        return bits.astype(np.uint16)
    return bits.view(np.float32 if dtype == "f32" else np.float16)


def oracle_layout(op, xs, attrs, dtype):
    """The oracle's layout primitive on the exact input values."""
    x64 = [bits_to_f64(b, dtype) for b in xs]
    if op == "transpose":
        return P.transpose(x64[0], attrs["perm"])
    if op == "slice":
        return P.slice_(x64[0], attrs["begin"], attrs["end"])
    if op == "pad":
        return P.pad(x64[0], attrs["lo"], attrs["hi"], attrs.get("value", 0.0))
    if op == "concat":
        parts = list(x64)
        if attrs.get("fill") is not None:
            shp = list(parts[-1].shape)
            shp[attrs["axis"]] = 1
            parts.append(P.fill(shp, attrs["fill"]))
        return P.concat(parts, attrs["axis"])
    raise ValueError(op)


@pytest.mark.parametrize("case", range(len(STANDALONE)))
def test_standalone_layout_kernel_bit_exact(case):
    from paper_2406_09465_amd import graphs
    from paper_2406_09465_amd.runner import PlanRunner
    op, dtype, shapes, attrs = STANDALONE[case]
    print(f"\n[case] layout stand-alone {op} {dtype} {shapes} {attrs}", flush=True)
    w = graphs.layout_probe(op, dtype, shapes, **attrs)
    xs = [probe_input(7000 + 10 * case + i, sh, dtype) for i, sh in enumerate(shapes)]
    r = PlanRunner(w, "unfused")
    r.set_inputs({f"in{i}": _raw_from_bits(b, dtype) for i, b in enumerate(xs)})
    r.launch()
    torch.cuda.synchronize()
    got = device_bits(r.outs[0])
    want64 = oracle_layout(op, xs, dict(attrs), dtype)
    want = to_storage_bits(want64, dtype).reshape(got.shape)
    # NaN inputs: the oracle carries NaN through float64, whose rounding back
    # gives the canonical quiet NaN, the same pattern the inputs hold
    assert_bits_equal(got, want, f"{op} {dtype} {shapes}")
