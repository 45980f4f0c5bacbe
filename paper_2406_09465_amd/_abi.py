"""ctypes binding of libkorch.so (include/korch.h): argument marshalling only.

Every computation happens in the library and its gfx950 kernels.  Importing
this module loads the in-tree ``libkorch.so`` and raises ``ImportError`` when it
is missing; nothing here falls back to another implementation.
"""

from __future__ import annotations

import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libkorch.so")

# Code objects compiled at run time are cached next to the package unless the
# caller chose another directory.
os.environ.setdefault("KORCH_CACHE_DIR", os.path.join(PKG, "_kcache"))

# KORCH_LIB loads another build of the library instead (e.g. one built with a
# host-code sanitizer).
LIB_PATH = os.environ.get("KORCH_LIB") or LIB_PATH
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2406_09465_amd.build`")
# A process must hold one HIP runtime.  PyTorch ships its own copy; loading it
# first lets the library's HIP dependencies resolve to that copy by soname.
# Loaded the other way round, the process would hold two HIP runtimes and the
# second to start would see no device.
try:
    import torch  # noqa: F401
except ImportError:
    pass
lib = C.CDLL(LIB_PATH)

MAX_RANK = 8
F32, F16, BF16 = 0, 1, 2
DTYPES = {"f32": F32, "f16": F16, "bf16": BF16}
DTYPE_NAMES = {v: k for k, v in DTYPES.items()}

OPS = {
    "input": 0,
    "neg": 1, "exp": 2, "log": 3, "tanh": 4, "sqrt": 5, "rsqrt": 6, "relu": 7, "square": 8, "recip": 9,
    "gelu_tanh": 10, "abs": 11, "identity": 12,
    "add": 32, "sub": 33, "mul": 34, "div": 35, "max": 36, "min": 37,
    "reduce_sum": 64, "reduce_mean": 65, "reduce_max": 66, "broadcast": 67,
    "transpose": 96, "reshape": 97, "slice": 98, "pad": 99, "concat": 100,
    "fill": 101,
    "matmul": 128, "conv2d": 129,
}
OP_NAMES = {v: k for k, v in OPS.items()}
# primitive-graph transformation rules (korch_rewrite_rule)
RW_DEFER_DIV, RW_REDUCE_AS_PRODUCT, RW_MERGE_PRODUCTS, RW_FOLD_SCALE, RW_ALL = 1, 2, 4, 8, 47
RW_LAYOUT_VARIANTS, RW_SPLIT_MOMENTS = 16, 32
FAMILIES = {0: "none", 1: "pointwise", 2: "row", 3: "colreduce", 4: "gemm", 5: "conv", 6: "attention", 7: "splitk"}

E_UNSUPPORTED = -20
E_COMPILE = -23


class korch_attrs(C.Structure):
    _fields_ = [
        ("axis", C.c_int32), ("keepdim", C.c_int32), ("rank", C.c_int32),
        ("perm", C.c_int32 * MAX_RANK), ("shape", C.c_int64 * MAX_RANK),
        ("begin", C.c_int64 * MAX_RANK), ("end", C.c_int64 * MAX_RANK),
        ("scalar", C.c_double), ("has_scalar", C.c_int32),
        ("stride", C.c_int32), ("pad", C.c_int32), ("pad_value", C.c_double),
    ]


class korch_kernel_desc(C.Structure):
    _fields_ = [("n_prims", C.c_int32), ("prims", C.POINTER(C.c_int32)),
                ("n_outs", C.c_int32), ("outs", C.POINTER(C.c_int32))]


_P = C.c_void_p
_I = C.c_int32
STATE_CB = C.CFUNCTYPE(C.c_int, C.POINTER(C.c_uint8), C.c_int32, C.c_void_p)
CAND_CB = C.CFUNCTYPE(C.c_int, C.POINTER(korch_kernel_desc), C.c_void_p)

_SIGS = {
    "korch_last_error": ([], C.c_char_p),
    "korch_status_name": ([C.c_int], C.c_char_p),
    "korch_graph_create": ([C.POINTER(_P)], C.c_int),
    "korch_graph_destroy": ([_P], None),
    "korch_graph_input": ([_P, _I, _I, C.POINTER(C.c_int64), C.POINTER(_I)], C.c_int),
    "korch_graph_op": ([_P, _I, _I, C.POINTER(_I), C.POINTER(korch_attrs), _I, C.POINTER(_I)], C.c_int),
    "korch_graph_output": ([_P, _I], C.c_int),
    "korch_graph_finalize": ([_P], C.c_int),
    "korch_graph_num_nodes": ([_P, C.POINTER(_I)], C.c_int),
    "korch_graph_node_info": ([_P, _I, C.POINTER(_I), C.POINTER(_I), C.POINTER(_I), C.POINTER(C.c_int64)], C.c_int),
    "korch_graph_node_inputs": ([_P, _I, C.POINTER(_I), _I, C.POINTER(_I)], C.c_int),
    "korch_graph_num_inputs": ([_P, C.POINTER(_I)], C.c_int),
    "korch_graph_num_outputs": ([_P, C.POINTER(_I)], C.c_int),
    "korch_graph_input_node": ([_P, _I, C.POINTER(_I)], C.c_int),
    "korch_graph_output_node": ([_P, _I, C.POINTER(_I)], C.c_int),
    "korch_is_convex": ([_P, _I, C.POINTER(_I), C.POINTER(_I)], C.c_int),
    "korch_enumerate_states": ([_P, _I, STATE_CB, _P], C.c_int),
    "korch_enumerate_candidates": ([_P, _I, _I, _I, CAND_CB, _P], C.c_int),
    "korch_kernel_family": ([_P, C.POINTER(korch_kernel_desc), C.POINTER(_I)], C.c_int),
    "korch_plan_create": ([_P, _I, C.POINTER(korch_kernel_desc), C.POINTER(_P)], C.c_int),
    "korch_plan_unfused": ([_P, C.POINTER(_P)], C.c_int),
    "korch_plan_destroy": ([_P], None),
    "korch_plan_num_kernels": ([_P, C.POINTER(_I)], C.c_int),
    "korch_plan_compile": ([_P], C.c_int),
    "korch_plan_load": ([_P], C.c_int),
    "korch_plan_workspace_bytes": ([_P, C.POINTER(C.c_size_t)], C.c_int),
    "korch_plan_execute": ([_P, C.POINTER(_P), C.POINTER(_P), _P, C.c_size_t, _P], C.c_int),
    "korch_plan_execute_noalloc": ([_P, C.POINTER(_P), C.POINTER(_P), _P], C.c_int),
    "korch_flush_caches": ([_P, C.c_size_t, _I, _P], C.c_int),
    "korch_plan_execute_events": ([_P, C.POINTER(_P), C.POINTER(_P), _P, C.c_size_t, _P, C.POINTER(_P), C.POINTER(_P)],
                                  C.c_int),
    "korch_plan_execute_kernels": ([_P, _I, _I, C.POINTER(_P), C.POINTER(_P), _P, C.c_size_t, _P], C.c_int),
    "korch_kernel_source": ([_P, _P, C.c_char_p, C.c_size_t, C.POINTER(C.c_size_t)], C.c_int),
    "korch_plan_kernel_code": ([_P, _I, _P, C.c_size_t, C.POINTER(C.c_size_t)], C.c_int),
    "korch_plan_execute_timed": ([_P, _I, _I, C.POINTER(_P), C.POINTER(_P), _P, C.c_size_t, _P, _I, _P, _P], C.c_int),
    "korch_plan_kernel_info": ([_P, _I, C.POINTER(_I), C.POINTER(C.c_double), C.POINTER(C.c_double)], C.c_int),
    "korch_plan_kernel_source": ([_P, _I, C.c_char_p, C.c_size_t, C.POINTER(C.c_size_t)], C.c_int),
    "korch_plan_kernel_name": ([_P, _I, C.c_char_p, C.c_size_t], C.c_int),
    "korch_plan_kernel_launch": ([_P, _I, C.POINTER(_I), C.POINTER(_I), C.POINTER(_I)], C.c_int),
    "korch_graph_node_attrs": ([_P, _I, C.POINTER(korch_attrs)], C.c_int),
    "korch_graph_rewrite": ([_P, C.c_uint32, C.POINTER(_P), C.POINTER(_I)], C.c_int),
    "korch_compile_candidate": ([_P, C.POINTER(korch_kernel_desc)], C.c_int),
    "korch_profile_candidate": ([_P, C.POINTER(korch_kernel_desc), _I, _I, C.c_size_t, _P, C.POINTER(C.c_float)],
                                C.c_int),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_SIGS)


class KorchError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{lib.korch_status_name(code).decode()} ({code}): {msg}")
        self.code = code


def check(rc):
    if rc != 0:
        raise KorchError(rc, lib.korch_last_error().decode())
    return rc


def _ids(xs):
    xs = [int(x) for x in xs]
    return (C.c_int32 * max(1, len(xs)))(*xs), len(xs)


def pointer_array(ptrs):
    """ctypes array of device pointers (ints), for the execute calls."""
    return (C.c_void_p * max(1, len(ptrs)))(*[C.c_void_p(int(p)) for p in ptrs])


def kernel_desc(prims, outs):
    """Build a korch_kernel_desc; returns (desc, keepalive)."""
    p, np_ = _ids(sorted(prims))
    o, no = _ids(sorted(outs))
    d = korch_kernel_desc(np_, C.cast(p, C.POINTER(C.c_int32)), no, C.cast(o, C.POINTER(C.c_int32)))
    return d, (p, o)


class Graph:
    """Primitive graph handle (korch_graph_*)."""

    def __init__(self):
        self.h = _P()
        check(lib.korch_graph_create(C.byref(self.h)))

    def __del__(self):
        if getattr(self, "h", None) and lib is not None:
            lib.korch_graph_destroy(self.h)
            self.h = None

    def input(self, dtype, shape):
        shape = [int(s) for s in shape]
        arr = (C.c_int64 * max(1, len(shape)))(*shape)
        node = _I()
        check(lib.korch_graph_input(self.h, DTYPES[dtype], len(shape), arr, C.byref(node)))
        return node.value

    def op(self, op, inputs, dtype, *, axis=0, keepdim=True, perm=None, shape=None, begin=None, end=None,
           scalar=None, stride=1, pad=0, pad_value=0.0):
        a = korch_attrs()
        a.axis = int(axis)
        a.keepdim = 1 if keepdim else 0
        seq = perm if perm is not None else (shape if shape is not None else (begin if begin is not None else ()))
        a.rank = len(seq)
        for i, v in enumerate(perm or ()):
            a.perm[i] = int(v)
        for i, v in enumerate(shape or ()):
            a.shape[i] = int(v)
        for i, v in enumerate(begin or ()):
            a.begin[i] = int(v)
        for i, v in enumerate(end or ()):
            a.end[i] = int(v)
        if scalar is not None:
            a.scalar = float(scalar)
            a.has_scalar = 1
        a.stride, a.pad, a.pad_value = int(stride), int(pad), float(pad_value)
        ids, n = _ids(inputs)
        node = _I()
        check(lib.korch_graph_op(self.h, OPS[op], n, ids, C.byref(a), DTYPES[dtype], C.byref(node)))
        return node.value

    def output(self, node):
        check(lib.korch_graph_output(self.h, int(node)))

    def finalize(self):
        check(lib.korch_graph_finalize(self.h))
        return self

    def num_nodes(self):
        n = _I()
        check(lib.korch_graph_num_nodes(self.h, C.byref(n)))
        return n.value

    def node_attrs(self, node):
        """Attributes of a node (as a dict; the reduce / concat axis normalized)."""
        a = korch_attrs()
        check(lib.korch_graph_node_attrs(self.h, int(node), C.byref(a)))
        r = a.rank
        return dict(axis=a.axis, keepdim=bool(a.keepdim), perm=tuple(a.perm[i] for i in range(r)),
                    shape=tuple(a.shape[i] for i in range(r)), begin=tuple(a.begin[i] for i in range(r)),
                    end=tuple(a.end[i] for i in range(r)), scalar=a.scalar if a.has_scalar else None,
                    value=a.scalar, stride=a.stride, pad=a.pad, pad_value=a.pad_value)

    def rewrite(self, rules=RW_ALL):
        """New graph after the primitive-graph transformations; (graph, applications)."""
        h, n = _P(), _I()
        check(lib.korch_graph_rewrite(self.h, int(rules), C.byref(h), C.byref(n)))
        g = Graph.__new__(Graph)
        g.h = h
        return g, n.value

    def node_info(self, node):
        op, dt, rank = _I(), _I(), _I()
        shape = (C.c_int64 * MAX_RANK)()
        check(lib.korch_graph_node_info(self.h, int(node), C.byref(op), C.byref(dt), C.byref(rank), shape))
        return OP_NAMES[op.value], DTYPE_NAMES[dt.value], tuple(shape[i] for i in range(rank.value))

    def node_inputs(self, node):
        n = _I()
        check(lib.korch_graph_node_inputs(self.h, int(node), None, 0, C.byref(n)))
        buf = (_I * max(1, n.value))()
        check(lib.korch_graph_node_inputs(self.h, int(node), buf, n.value, C.byref(n)))
        return [buf[i] for i in range(n.value)]

    def inputs(self):
        n = _I()
        check(lib.korch_graph_num_inputs(self.h, C.byref(n)))
        out = []
        for i in range(n.value):
            v = _I()
            check(lib.korch_graph_input_node(self.h, i, C.byref(v)))
            out.append(v.value)
        return out

    def outputs(self):
        n = _I()
        check(lib.korch_graph_num_outputs(self.h, C.byref(n)))
        out = []
        for i in range(n.value):
            v = _I()
            check(lib.korch_graph_output_node(self.h, i, C.byref(v)))
            out.append(v.value)
        return out

    def is_convex(self, nodes):
        ids, n = _ids(nodes)
        r = _I()
        check(lib.korch_is_convex(self.h, n, ids, C.byref(r)))
        return bool(r.value)

    def states(self, max_states=100000):
        out = []

        def cb(mem, n, user):
            out.append(frozenset(i for i in range(n) if mem[i]))
            return 0

        f = STATE_CB(cb)
        check(lib.korch_enumerate_states(self.h, int(max_states), f, None))
        return out

    def candidates(self, max_prims=64, max_outs=3, only_supported=False, limit=None):
        out = []

        def cb(d, user):
            dd = d.contents
            out.append((tuple(dd.prims[i] for i in range(dd.n_prims)), tuple(dd.outs[i] for i in range(dd.n_outs))))
            return 1 if (limit is not None and len(out) >= limit) else 0

        f = CAND_CB(cb)
        check(lib.korch_enumerate_candidates(self.h, int(max_prims), int(max_outs), 1 if only_supported else 0, f,
                                             None))
        return out

    def family(self, prims, outs):
        d, keep = kernel_desc(prims, outs)
        fam = _I()
        check(lib.korch_kernel_family(self.h, C.byref(d), C.byref(fam)))
        return FAMILIES[fam.value]

    def kernel_source(self, prims, outs):
        """HIP source generated for kernel (prims, outs) within this graph."""
        d, keep = kernel_desc(prims, outs)
        n = C.c_size_t()
        check(lib.korch_kernel_source(self.h, C.byref(d), None, 0, C.byref(n)))
        buf = C.create_string_buffer(n.value + 1)
        check(lib.korch_kernel_source(self.h, C.byref(d), buf, n.value + 1, None))
        return buf.value.decode()

    def compile_candidate(self, prims, outs):
        """Compiles the single kernel (prims, outs) as the profiler will; False when unsupported."""
        d, keep = kernel_desc(prims, outs)
        rc = lib.korch_compile_candidate(self.h, C.byref(d))
        if rc == E_UNSUPPORTED:
            return False
        check(rc)
        return True

    def profile(self, prims, outs, warmup=20, reps=100, flush_bytes=512 << 20, stream=0):
        """Median latency (us) of the single kernel (prims, outs); None when unsupported (infinite cost)."""
        d, keep = kernel_desc(prims, outs)
        us = C.c_float()
        rc = lib.korch_profile_candidate(self.h, C.byref(d), int(warmup), int(reps), int(flush_bytes),
                                         C.c_void_p(stream), C.byref(us))
        if rc == E_UNSUPPORTED:
            return None
        check(rc)
        return us.value


class Plan:
    """Orchestration plan handle (korch_plan_*)."""

    def __init__(self, graph: Graph, kernels=None):
        self.h = _P()
        self.graph = graph
        if kernels is None:
            check(lib.korch_plan_unfused(graph.h, C.byref(self.h)))
        else:
            descs = (korch_kernel_desc * max(1, len(kernels)))()
            keep = []
            for i, (prims, outs) in enumerate(kernels):
                d, k = kernel_desc(prims, outs)
                descs[i] = d
                keep.append(k)
            check(lib.korch_plan_create(graph.h, len(kernels), descs, C.byref(self.h)))

    def __del__(self):
        if getattr(self, "h", None) and lib is not None:
            lib.korch_plan_destroy(self.h)
            self.h = None

    def num_kernels(self):
        n = _I()
        check(lib.korch_plan_num_kernels(self.h, C.byref(n)))
        return n.value

    def compile(self):
        check(lib.korch_plan_compile(self.h))
        return self

    def load(self):
        check(lib.korch_plan_load(self.h))
        return self

    def workspace_bytes(self):
        n = C.c_size_t()
        check(lib.korch_plan_workspace_bytes(self.h, C.byref(n)))
        return n.value

    def execute(self, inputs, outputs, workspace=0, workspace_bytes=0, stream=0):
        """inputs / outputs: device pointers (ints) in graph input / output order, or
        ctypes pointer arrays already built with ``pointer_array``."""
        ins = inputs if isinstance(inputs, C.Array) else pointer_array(inputs)
        outs = outputs if isinstance(outputs, C.Array) else pointer_array(outputs)
        check(lib.korch_plan_execute(self.h, ins, outs, C.c_void_p(int(workspace)), int(workspace_bytes),
                                     C.c_void_p(int(stream))))

    def execute_noalloc(self, inputs, outputs, stream=0):
        """korch_plan_execute_noalloc: workspace and counters in the library's
        static device scratch (no allocation; the plan must be loaded)."""
        ins = inputs if isinstance(inputs, C.Array) else pointer_array(inputs)
        outs = outputs if isinstance(outputs, C.Array) else pointer_array(outputs)
        check(lib.korch_plan_execute_noalloc(self.h, ins, outs, C.c_void_p(int(stream))))

    def execute_kernels(self, first, count, inputs, outputs, workspace=0, workspace_bytes=0, stream=0):
        ins = inputs if isinstance(inputs, C.Array) else pointer_array(inputs)
        outs = outputs if isinstance(outputs, C.Array) else pointer_array(outputs)
        check(lib.korch_plan_execute_kernels(self.h, int(first), int(count), ins, outs, C.c_void_p(int(workspace)),
                                             int(workspace_bytes), C.c_void_p(int(stream))))

    def execute_timed(self, first, count, inputs, outputs, workspace=0, workspace_bytes=0, stream=0, timed=0,
                      start=0, stop=0):
        """execute_kernels with kernel ``timed`` bracketed by the hipEvent_t handles ``start`` / ``stop``.
        ``inputs`` / ``outputs`` may be ctypes pointer arrays already built (see ``pointer_array``)."""
        ins = inputs if isinstance(inputs, C.Array) else pointer_array(inputs)
        outs = outputs if isinstance(outputs, C.Array) else pointer_array(outputs)
        check(lib.korch_plan_execute_timed(self.h, int(first), int(count), ins, outs, C.c_void_p(int(workspace)),
                                           int(workspace_bytes), C.c_void_p(int(stream)), int(timed),
                                           C.c_void_p(int(start)), C.c_void_p(int(stop))))

    def kernel_info(self, k):
        fam, b, f = _I(), C.c_double(), C.c_double()
        check(lib.korch_plan_kernel_info(self.h, int(k), C.byref(fam), C.byref(b), C.byref(f)))
        return FAMILIES[fam.value], b.value, f.value

    def kernel_source(self, k):
        n = C.c_size_t()
        check(lib.korch_plan_kernel_source(self.h, int(k), None, 0, C.byref(n)))
        buf = C.create_string_buffer(n.value + 1)
        check(lib.korch_plan_kernel_source(self.h, int(k), buf, n.value + 1, None))
        return buf.value.decode()

    def kernel_code(self, k):
        """The compiled gfx950 code object (ELF bytes) of kernel k."""
        n = C.c_size_t()
        check(lib.korch_plan_kernel_code(self.h, int(k), None, 0, C.byref(n)))
        buf = C.create_string_buffer(max(n.value, 1))
        check(lib.korch_plan_kernel_code(self.h, int(k), buf, n.value, None))
        return buf.raw[:n.value]

    def kernel_name(self, k):
        buf = C.create_string_buffer(256)
        check(lib.korch_plan_kernel_name(self.h, int(k), buf, 256))
        return buf.value.decode()

    def kernel_launch(self, k):
        g, b, lds = (_I * 3)(), (_I * 3)(), _I()
        check(lib.korch_plan_kernel_launch(self.h, int(k), g, b, C.byref(lds)))
        return tuple(g), tuple(b), lds.value
