"""Primitive graph container, shape rules, unfused executor and plan executor.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A primitive graph G = (P, E) is a DAG: nodes are primitives, an edge (p1, p2)
is a tensor produced by p1 and read by p2 (Korch, Section 4).  Graph inputs
(activations and weights alike) are nodes with no producer.

Plan semantics (Section 4, "Kernel orchestration problem"; Section 5.3):
  * a kernel is a pair (P', O): a set of primitives P' and the subset O of
    P' whose tensors it materializes;
  * a kernel reads, for every edge (u, v) with v in P' and u outside P', the
    materialized tensor of u; kernels run one after another in list order;
  * a primitive may be executed by several kernels (redundant execution) and a
    primitive in no kernel is simply never executed (implicit pruning).
A contiguous reshape only reinterprets an existing tensor, so the reshape of a
materialized tensor is itself available without any kernel.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import primitives as prim

ELEMENTWISE_UNARY = set(prim.UNARY)
ELEMENTWISE_BINARY = set(prim.BINARY)
REDUCE = {"reduce_sum", "reduce_mean", "reduce_max"}
LAYOUT = {"transpose", "reshape", "slice", "pad", "concat"}
LINEAR = {"matmul", "conv2d"}


@dataclass
class Node:
    name: str
    op: str                      # "input" or a primitive name
    inputs: tuple = ()
    attrs: dict = field(default_factory=dict)
    shape: tuple = ()
    dtype: str = "f32"


def _broadcast_shapes(a, b):
    r = max(len(a), len(b))
    a = (1,) * (r - len(a)) + tuple(a)
    b = (1,) * (r - len(b)) + tuple(b)
    out = []
    for x, y in zip(a, b):
        if x != y and x != 1 and y != 1:
            raise ValueError(f"shapes {a} and {b} do not broadcast")
        out.append(max(x, y))
    return tuple(out)


class Graph:
    """A DAG of primitives in creation order (every node's inputs precede it)."""

    def __init__(self, dtype="f32"):
        self.nodes: list[Node] = []
        self.outputs: list[int] = []
        self.dtype = dtype

    # -- construction ------------------------------------------------------
    def input(self, name, shape, dtype=None):
        self.nodes.append(Node(name, "input", (), {}, tuple(int(s) for s in shape), dtype or self.dtype))
        return len(self.nodes) - 1

    def op(self, op, inputs, name=None, **attrs):
        inputs = tuple(int(i) for i in inputs)
        dtype = attrs.pop("dtype", None) or self.dtype
        for i in inputs:
            if not 0 <= i < len(self.nodes):
                raise ValueError("input refers to a later or missing node")
        shape = self._infer(op, inputs, attrs)
        name = name or f"{op}{len(self.nodes)}"
        self.nodes.append(Node(name, op, inputs, dict(attrs), shape, dtype))
        return len(self.nodes) - 1

    def output(self, i):
        self.outputs.append(int(i))

    def index(self, name):
        for i, n in enumerate(self.nodes):
            if n.name == name:
                return i
        raise KeyError(name)

    # -- shape rules -------------------------------------------------------
    def _infer(self, op, inputs, a):
        sh = [self.nodes[i].shape for i in inputs]
        if op in ELEMENTWISE_UNARY:
            return sh[0]
        if op in ELEMENTWISE_BINARY:
            return sh[0] if len(sh) == 1 else _broadcast_shapes(sh[0], sh[1])
        if op in REDUCE:
            ax = a["axis"] % len(sh[0])
            if a.get("keepdim", True):
                return sh[0][:ax] + (1,) + sh[0][ax + 1:]
            return sh[0][:ax] + sh[0][ax + 1:]
        if op == "broadcast":
            _broadcast_shapes(sh[0], a["shape"])
            return tuple(a["shape"])
        if op == "transpose":
            return tuple(sh[0][p] for p in a["perm"])
        if op == "reshape":
            if int(np.prod(a["shape"])) != int(np.prod(sh[0])):
                raise ValueError("reshape changes the element count")
            return tuple(a["shape"])
        if op == "slice":
            return tuple(int(e) - int(b) for b, e in zip(a["begin"], a["end"]))
        if op == "pad":
            return tuple(s + int(l) + int(h) for s, l, h in zip(sh[0], a["lo"], a["hi"]))
        if op == "fill":
            return tuple(int(d) for d in a["shape"])
        if op == "concat":
            ax = a["axis"]
            out = list(sh[0])
            out[ax] = sum(s[ax] for s in sh)
            return tuple(out)
        if op == "matmul":
            x, y = sh
            if x[-1] != y[-2]:
                raise ValueError("contraction sizes differ")
            batch = _broadcast_shapes(x[:-2], y[:-2])
            return batch + (x[-2], y[-1])
        if op == "conv2d":
            x, w = sh
            s, p = a.get("stride", 1), a.get("pad", 0)
            kh, kw, cin, cout = w
            ho = (x[-3] + 2 * p - kh) // s + 1
            wo = (x[-2] + 2 * p - kw) // s + 1
            return x[:-3] + (ho, wo, cout)
        raise ValueError(f"unknown primitive {op}")

    # -- structure ---------------------------------------------------------
    def consumers(self):
        cons = [[] for _ in self.nodes]
        for v, n in enumerate(self.nodes):
            for u in n.inputs:
                cons[u].append(v)
        return cons

    def primitives(self):
        return [i for i, n in enumerate(self.nodes) if n.op != "input"]

    def edges(self):
        return [(u, v) for v, n in enumerate(self.nodes) for u in n.inputs]


# ----------------------------------------------------------------------------
# Execution
# ----------------------------------------------------------------------------


def evaluate_node(g: Graph, i: int, args):
    """Run primitive ``i`` on float64 operand arrays ``args`` (one per input)."""
    n = g.nodes[i]
    op, a = n.op, n.attrs
    if op in ELEMENTWISE_UNARY or op in ELEMENTWISE_BINARY:
        return prim.elementwise(op, args, a.get("scalar"))
    if op in REDUCE:
        return prim.reduce(op, args[0], a["axis"], a.get("keepdim", True))
    if op == "broadcast":
        return prim.broadcast(args[0], a["shape"])
    if op == "transpose":
        return prim.transpose(args[0], a["perm"])
    if op == "reshape":
        return prim.reshape(args[0], a["shape"])
    if op == "slice":
        return prim.slice_(args[0], a["begin"], a["end"])
    if op == "pad":
        return prim.pad(args[0], a["lo"], a["hi"], a.get("value", 0.0))
    if op == "concat":
        return prim.concat(args, a["axis"])
    if op == "fill":
        return prim.fill(a["shape"], a["value"])
    if op == "matmul":
        return prim.matmul(args[0], args[1])
    if op == "conv2d":
        return prim.conv2d_nhwc(args[0], args[1], a.get("stride", 1), a.get("pad", 0))
    raise ValueError(f"unknown primitive {op}")


def _round_like_storage(x, dtype):
    if dtype == "f16":
        return x.astype(np.float16).astype(np.float64)
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        from synthetic import bf16_bits_to_f32, f32_to_bf16_bits
        return bf16_bits_to_f32(f32_to_bf16_bits(x.astype(np.float32))).astype(np.float64)
    return x


def run_unfused(g: Graph, inputs: dict, round_storage: bool = False, keep_all: bool = False):
    """Execute every primitive once, in creation (topological) order.

    ``inputs`` maps input names to float64 arrays.  Returns ``{name: array}``
    for the graph outputs (or for every node when ``keep_all``).
    ``round_storage`` is a diagnostic mode that rounds every node's output to
    its storage dtype, as a one-kernel-per-primitive GPU run would store it.
    """
    vals = {}
    for i, n in enumerate(g.nodes):
        if n.op == "input":
            v = np.asarray(inputs[n.name], dtype=np.float64)
            if v.shape != n.shape:
                raise ValueError(f"input {n.name}: shape {v.shape} != {n.shape}")
            vals[i] = v
            continue
        v = evaluate_node(g, i, [vals[u] for u in n.inputs])
        if round_storage:
            v = _round_like_storage(v, n.dtype)
        vals[i] = v
    keys = range(len(g.nodes)) if keep_all else g.outputs
    return {g.nodes[i].name: vals[i] for i in keys}


class PlanError(Exception):
    pass


def run_plan(g: Graph, plan, inputs: dict):
    """Execute an orchestration plan: a list of kernels ``(prims, outs)``.

    Each kernel computes its primitives from the tensors materialized by
    earlier kernels (or graph inputs), and materializes only ``outs``.  Raises
    ``PlanError`` when a kernel needs a tensor nobody materialized or when a
    graph output is never materialized.
    """
    mat = {}
    for i, n in enumerate(g.nodes):
        if n.op == "input":
            mat[i] = np.asarray(inputs[n.name], dtype=np.float64)

    def available(u):
        if u in mat:
            return mat[u]
        n = g.nodes[u]
        if n.op == "reshape":
            src = available(n.inputs[0])
            if src is not None:
                return prim.reshape(src, n.attrs["shape"])
        return None

    for kprims, kouts in plan:
        kset = set(kprims)
        local = {}
        for i in sorted(kset):
            n = g.nodes[i]
            if n.op == "input":
                raise PlanError("a kernel may not contain a graph input")
            args = []
            for u in n.inputs:
                if u in kset:
                    args.append(local[u])
                else:
                    v = available(u)
                    if v is None:
                        raise PlanError(f"kernel reads {g.nodes[u].name}, which no earlier kernel materialized")
                    args.append(v)
            local[i] = evaluate_node(g, i, args)
        for o in kouts:
            if o not in kset:
                raise PlanError("an output is not in its kernel")
            mat[o] = local[o]
    out = {}
    for o in g.outputs:
        v = available(o)
        if v is None:
            raise PlanError(f"graph output {g.nodes[o].name} is never materialized")
        out[g.nodes[o].name] = v
    return out
