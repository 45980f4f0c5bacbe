"""Primitive graphs of the five workloads, built through the C ABI, with their plans.

Operator fission is applied by hand (Korch, Section 3): softmax becomes a row
max, a subtraction, an exponential, a row sum and a division; LayerNorm
becomes mean, subtraction, square, mean, add-eps, reciprocal square root,
scaling and the affine pair; Mish becomes exp, add 1, log, tanh and a product.
Broadcast is implicit in binary primitives (ONNX style, Section 5.1).

Each builder returns a ``Workload`` with the graph handle, a name -> node map,
and named plans:
  * "fused":   the recommended orchestration (fewest kernels, redundant
               recomputation where it saves traffic: Section 4.2);
  * "layered": a plan that keeps each dense product in its own kernel;
  * "unfused": one kernel per primitive (korch_plan_unfused).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

from ._abi import Graph, Plan


@dataclass
class Workload:
    name: str
    dtype: str
    graph: Graph
    ids: dict
    input_names: list
    output_names: list
    plans: dict = field(default_factory=dict)  # name -> list of (prim names, out names)
    sizes: dict = field(default_factory=dict)

    def node(self, name):
        return self.ids[name]

    def kernels(self, plan_name):
        ks = []
        for prims, outs in self.plans[plan_name]:
            ks.append(([self.ids[p] for p in prims], [self.ids[o] for o in outs]))
        return ks

    def plan(self, plan_name):
        if plan_name == "unfused":
            return Plan(self.graph)
        return Plan(self.graph, self.kernels(plan_name))


class _B:
    """Small helper that names nodes as they are created."""

    def __init__(self, dtype):
        self.g = Graph()
        self.dtype = dtype
        self.ids = {}
        self.inputs = []

    def inp(self, name, shape):
        self.ids[name] = self.g.input(self.dtype, shape)
        self.inputs.append(name)
        return self.ids[name]

    def op(self, name, op, ins, **attrs):
        self.ids[name] = self.g.op(op, [self.ids[i] for i in ins], self.dtype, **attrs)
        return self.ids[name]


def _finish(b, name, outputs, sizes, extra_outputs=()):
    """Marks the outputs (then any extra named nodes, so that a test can read
    an intermediate tensor of the unfused plan) and finalizes the graph."""
    names = list(outputs) + [x for x in extra_outputs if x not in outputs]
    for o in names:
        b.g.output(b.ids[o])
    b.g.finalize()
    return Workload(name, b.dtype, b.g, b.ids, b.inputs, names, sizes=sizes)


def _softmax(b, s):
    b.op("m", "reduce_max", [s], axis=-1, keepdim=True)
    b.op("Z", "sub", [s, "m"])
    b.op("E", "exp", ["Z"])
    b.op("s", "reduce_sum", ["E"], axis=-1, keepdim=True)
    b.op("P", "div", ["E", "s"])


def _layernorm(b, x, eps, p=""):
    b.op(p + "mu", "reduce_mean", [x], axis=-1, keepdim=True)
    b.op(p + "D", "sub", [x, p + "mu"])
    b.op(p + "D2", "square", [p + "D"])
    b.op(p + "var", "reduce_mean", [p + "D2"], axis=-1, keepdim=True)
    b.op(p + "ve", "add", [p + "var"], scalar=eps)
    b.op(p + "r", "rsqrt", [p + "ve"])
    b.op(p + "Xh", "mul", [p + "D", p + "r"])
    b.op(p + "Yg", "mul", [p + "Xh", "gamma"])
    b.op(p + "Y", "add", [p + "Yg", "beta"])
    return p + "Y"


def attention(n=128, d=64, nk=None, dtype="f32", extra_outputs=()):
    nk = n if nk is None else nk
    b = _B(dtype)
    b.inp("Q", (n, d))
    b.inp("K", (nk, d))
    b.inp("V", (nk, d))
    b.op("KT", "transpose", ["K"], perm=(1, 0))
    b.op("S0", "matmul", ["Q", "KT"])
    b.op("S", "mul", ["S0"], scalar=1.0 / math.sqrt(d))
    _softmax(b, "S")
    b.op("O", "matmul", ["P", "V"])
    w = _finish(b, "attention", ["O"], dict(n=n, d=d, nk=nk), extra_outputs)
    w.plans["fused"] = [(["KT", "S0", "S", "m", "Z", "E", "s", "P", "O"], ["O"])]
    w.plans["layered"] = [(["KT", "S0", "S"], ["S"]), (["m", "Z", "E", "s", "P"], ["P"]), (["O"], ["O"])]
    return w


def mlp(m=4096, d=768, h=3072, dtype="f16", eps=1e-5, extra_outputs=()):
    b = _B(dtype)
    b.inp("X", (m, d))
    b.inp("W1", (d, h))
    b.inp("W2", (h, d))
    b.inp("gamma", (d,))
    b.inp("beta", (d,))
    _layernorm(b, "X", eps)
    b.op("H0", "matmul", ["Y", "W1"])
    b.op("Hg", "gelu_tanh", ["H0"])
    b.op("Zo", "matmul", ["Hg", "W2"])
    b.op("out", "add", ["Zo", "X"])
    w = _finish(b, "mlp", ["out"], dict(m=m, d=d, h=h), extra_outputs)
    # The statistics kernel materializes the centred rows D and the row scale
    # r (two outputs); normalization and affine run in the first product's
    # operand prologue, GELU in its epilogue, the residual in the second
    # product's epilogue.  (mu cannot be an output of a kernel that also holds
    # its only consumer D: Definition 3.)
    w.plans["fused"] = [
        (["mu", "D", "D2", "var", "ve", "r"], ["D", "r"]),
        (["Xh", "Yg", "Y", "H0", "Hg"], ["Hg"]),
        (["Zo", "out"], ["out"]),
    ]
    w.plans["layered"] = [
        (["mu", "D", "D2", "var", "ve", "r", "Xh", "Yg", "Y"], ["Y"]),
        (["H0", "Hg"], ["Hg"]),
        (["Zo", "out"], ["out"]),
    ]
    return w


def sra(hh=128, ww=128, c=64, r=8, dtype="f16", eps=1e-5, extra_outputs=()):
    b = _B(dtype)
    b.inp("X", (hh, ww, c))
    b.inp("Wsr", (r * r * c, c))
    b.inp("gamma", (c,))
    b.inp("beta", (c,))
    b.op("Xr", "reshape", ["X"], shape=(hh // r, r, ww // r, r, c))
    b.op("Xt", "transpose", ["Xr"], perm=(0, 2, 1, 3, 4))
    b.op("A", "reshape", ["Xt"], shape=((hh // r) * (ww // r), r * r * c))
    b.op("KVp", "matmul", ["A", "Wsr"])
    kv = _layernorm(b, "KVp", eps, p="ln_")
    b.op("Qv", "reshape", ["X"], shape=(hh * ww, c))
    b.op("KT", "transpose", [kv], perm=(1, 0))
    b.op("S0", "matmul", ["Qv", "KT"])
    b.op("S", "mul", ["S0"], scalar=1.0 / math.sqrt(c))
    _softmax(b, "S")
    b.op("O", "matmul", ["P", kv])
    w = _finish(b, "sra", ["O"], dict(hh=hh, ww=ww, c=c, r=r), extra_outputs)
    ln = ["ln_mu", "ln_D", "ln_D2", "ln_var", "ln_ve", "ln_r", "ln_Xh", "ln_Yg", "ln_Y"]
    w.plans["fused"] = [
        (["Xt", "A", "KVp"] + ln, ["ln_Y"]),
        (["KT", "S0", "S", "m", "Z", "E", "s", "P", "O"], ["O"]),
    ]
    w.plans["layered"] = [
        (["Xt", "A", "KVp"], ["KVp"]),
        (ln, ["ln_Y"]),
        (["KT", "S0", "S"], ["S"]),
        (["m", "Z", "E", "s", "P"], ["P"]),
        (["O"], ["O"]),
    ]
    return w


def conv(hh=416, ww=416, cin=32, cout=64, k=3, dtype="f16", extra_outputs=()):
    b = _B(dtype)
    b.inp("X", (hh, ww, cin))
    b.inp("W", (k, k, cin, cout))
    b.inp("scale", (cout,))
    b.inp("shift", (cout,))
    b.op("C", "conv2d", ["X", "W"], stride=1, pad=k // 2)
    b.op("B1", "mul", ["C", "scale"])
    b.op("B", "add", ["B1", "shift"])
    b.op("E", "exp", ["B"])
    b.op("E1", "add", ["E"], scalar=1.0)
    b.op("SP", "log", ["E1"])
    b.op("T", "tanh", ["SP"])
    b.op("Y", "mul", ["B", "T"])
    w = _finish(b, "conv", ["Y"], dict(hh=hh, ww=ww, cin=cin, cout=cout, k=k), extra_outputs)
    w.plans["fused"] = [(["C", "B1", "B", "E", "E1", "SP", "T", "Y"], ["Y"])]
    w.plans["layered"] = [(["C", "B1", "B"], ["B"]), (["E", "E1", "SP", "T", "Y"], ["Y"])]
    return w


def linattn(heads=16, n=4096, d=16, dtype="bf16", eps=1e-6, extra_outputs=()):
    b = _B(dtype)
    b.inp("Q", (heads, n, d))
    b.inp("K", (heads, n, d))
    b.inp("V", (heads, n, d))
    b.op("Qr", "relu", ["Q"])
    b.op("Kr", "relu", ["K"])
    b.op("KrT", "transpose", ["Kr"], perm=(0, 2, 1))
    b.op("KVm", "matmul", ["KrT", "V"])
    b.op("sK", "reduce_sum", ["Kr"], axis=1, keepdim=True)
    b.op("num", "matmul", ["Qr", "KVm"])
    b.op("sKT", "transpose", ["sK"], perm=(0, 2, 1))
    b.op("den0", "matmul", ["Qr", "sKT"])
    b.op("den", "add", ["den0"], scalar=eps)
    b.op("out", "div", ["num", "den"])
    w = _finish(b, "linattn", ["out"], dict(heads=heads, n=n, d=d), extra_outputs)
    w.plans["fused"] = [
        (["Kr", "KrT", "KVm", "sK"], ["KVm", "sK"]),
        (["Qr", "num", "sKT", "den0", "den", "out"], ["out"]),
    ]
    w.plans["layered"] = [
        (["Kr", "KrT", "KVm"], ["KVm"]),
        (["Kr", "sK"], ["sK"]),
        (["Qr", "num", "sKT", "den0", "den", "out"], ["out"]),
    ]
    return w


def instnorm(hh=224, ww=224, c=32, dtype="f16", eps=1e-5, extra_outputs=()):
    b = _B(dtype)
    b.inp("X", (hh, ww, c))
    b.inp("gamma", (c,))
    b.inp("beta", (c,))
    b.op("Xp", "reshape", ["X"], shape=(hh * ww, c))
    b.op("mu", "reduce_mean", ["Xp"], axis=0, keepdim=True)
    b.op("D", "sub", ["Xp", "mu"])
    b.op("D2", "square", ["D"])
    b.op("var", "reduce_mean", ["D2"], axis=0, keepdim=True)
    b.op("ve", "add", ["var"], scalar=eps)
    b.op("r", "rsqrt", ["ve"])
    b.op("Xh", "mul", ["D", "r"])
    b.op("Yg", "mul", ["Xh", "gamma"])
    b.op("Y", "add", ["Yg", "beta"])
    b.op("R", "relu", ["Y"])
    b.op("Ri", "reshape", ["R"], shape=(hh, ww, c))
    b.op("out", "pad", ["Ri"], begin=(1, 1, 0), end=(1, 1, 0))
    w = _finish(b, "instnorm", ["out"], dict(hh=hh, ww=ww, c=c), extra_outputs)
    # operator per kernel (InstanceNorm as mean, variance and normalize; ReLU; Pad).
    # D feeds both the variance and the normalization, and a kernel holding D
    # and Xh but not the variance chain would not be convex, so the variance
    # kernel materializes D.
    w.plans["layered"] = [(["mu"], ["mu"]), (["D", "D2", "var", "ve", "r"], ["D", "r"]),
                          (["Xh", "Yg", "Y"], ["Y"]), (["R"], ["R"]), (["out"], ["out"])]
    # norm fission fused into the following ReLU and Pad (Section 6 case study)
    w.plans["fused"] = [(["mu"], ["mu"]), (["D", "D2", "var", "ve", "r"], ["D", "r"]),
                        (["Xh", "Yg", "Y", "R", "Ri", "out"], ["out"])]
    return w


def layout_probe(op, dtype, shapes, **attrs):
    """A graph of one layout primitive (transpose, slice, pad or concat) on
    graph inputs of the given shapes; a concat whose ``fill`` attribute is set
    appends a constant operand of that value (as the product-merging
    transformation does).  Its unfused plan is one kernel per primitive, the
    same generated kernels as the layout nodes of a workload's unfused plan."""
    b = _B(dtype)
    names = []
    for i, sh in enumerate(shapes):
        b.inp(f"in{i}", sh)
        names.append(f"in{i}")
    fill = attrs.pop("fill", None)
    if fill is not None:
        last = list(shapes[-1])
        last[attrs.get("axis", -1)] = 1
        b.op("ones", "fill", [], shape=tuple(last), scalar=fill)
        names.append("ones")
    if op == "pad":
        attrs = dict(begin=attrs["lo"], end=attrs["hi"], pad_value=attrs.get("value", 0.0))
    b.op("out", op, names, **attrs)
    return _finish(b, f"layout_{op}", ["out"], dict(shapes=[tuple(s) for s in shapes]))


BUILDERS = {"attention": attention, "mlp": mlp, "sra": sra, "conv": conv, "linattn": linattn, "instnorm": instnorm}


def rewritten(w: Workload, rules=None):
    """The workload's graph after the primitive-graph transformations
    (korch_graph_rewrite), with the same input and output names; returns
    (workload, number of rule applications).  It has no hand-written plans."""
    from ._abi import RW_ALL
    g2, n = w.graph.rewrite(RW_ALL if rules is None else rules)
    ids = dict(zip(w.input_names, g2.inputs()))
    ids.update(zip(w.output_names, g2.outputs()))
    return Workload(w.name, w.dtype, g2, ids, list(w.input_names), list(w.output_names), sizes=dict(w.sizes)), n


def moments_plan(w: Workload):
    """Two kernels for an InstanceNorm whose graph went through the
    split-moments transformation (its variance squares m - X, a node of its
    own): the column moments {mean, m - X, square, variance, + eps, rsqrt}
    exporting the mean and the reciprocal deviation (one pass over X), then
    everything else (X - m recomputed, the normalization and what follows).
    None when the graph has no such variance."""
    g = w.graph
    n = g.num_nodes()
    op = {v: g.node_info(v)[0] for v in range(n)}
    ins = {v: g.node_inputs(v) for v in range(n) if op[v] != "input"}
    cons = {v: [c for c in ins if v in ins[c]] for v in range(n)}
    for var in (v for v in range(n) if op[v] == "reduce_mean"):
        sq = ins[var][0]
        if op[sq] != "square" or op[ins[sq][0]] != "sub":
            continue
        dc = ins[sq][0]
        mu, x = ins[dc]
        if op[mu] != "reduce_mean" or ins[mu][0] != x:
            continue
        k0 = {mu, dc, sq, var}
        if op[x] == "reshape":
            k0.add(x)
        last = var
        while len(cons[last]) == 1 and op[cons[last][0]] in ("add", "rsqrt") and g.node_info(cons[last][0])[2] == g.node_info(var)[2]:
            last = cons[last][0]
            k0.add(last)
        prims = [v for v in range(n) if op[v] != "input"]
        return [(sorted(k0), sorted([mu, last])),
                (sorted(v for v in prims if v not in k0), sorted(o for o in g.outputs() if o not in k0))]
    return None


def plan_record(w: Workload, kernels, rules=0):
    """JSON-able record of a plan of ``w`` (or of its rewritten graph when
    ``rules`` is non-zero): node ids, plus names where the workload names them."""
    from ._abi import RW_LAYOUT_VARIANTS
    names = {v: k for k, v in w.ids.items()} if not rules else {}
    label = "original" if not rules else "layout variants" if rules == RW_LAYOUT_VARIANTS else "rewritten"
    return {"graph": label, "rules": int(rules),
            "kernel_ids": [[list(map(int, p)), list(map(int, o))] for p, o in kernels],
            "kernels": [[[names.get(v, f"#{v}") for v in p], [names.get(v, f"#{v}") for v in o]] for p, o in kernels]}


def plan_from_record(w: Workload, rec):
    """(workload, kernels) of a record written by plan_record."""
    if rec.get("rules"):
        w, _ = rewritten(w, rec["rules"])
    return w, [(list(p), list(o)) for p, o in rec["kernel_ids"]]


def build(workload: str, **sizes) -> Workload:
    return BUILDERS[workload](**sizes)
