"""Executes a compiled plan on torch device tensors (memory and streams only).

torch allocates device memory and supplies the stream; every primitive runs in
the library's generated gfx950 kernels.  There is no CPU fallback: running a
plan needs a GPU and the in-tree libkorch.so.
"""

from __future__ import annotations

import numpy as np
import torch

import ctypes as C

from ._abi import Plan, check, lib, pointer_array

TORCH_DTYPE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def to_device(arr: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Storage array (float32 / float16 / uint16 bf16 bits) -> device tensor of the same bytes."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr))
    return t.to(device)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


class PlanRunner:
    """A compiled plan plus device buffers for one workload instance."""

    def __init__(self, workload, plan="fused", kernels=None, device="cuda"):
        if not torch.cuda.is_available():
            raise RuntimeError("PlanRunner needs a GPU")
        self.w = workload
        self.device = device
        self.plan = Plan(workload.graph, kernels) if kernels is not None else workload.plan(plan)
        self.plan.compile()
        self.plan.load()  # code objects and the counter buffer on the current device
        self.ws_bytes = self.plan.workspace_bytes()
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device=device)
        g = workload.graph
        self.outs = []
        for o in g.outputs():
            _, dt, shape = g.node_info(o)
            self.outs.append(torch.empty(shape, dtype=TORCH_DTYPE[dt], device=device))
        self.ins = []

    def set_inputs(self, storage: dict):
        """storage: {input name: storage array} (synthetic.make_inputs output)."""
        self.ins = [to_device(storage[n], self.w.dtype, self.device) for n in self.w.input_names]

    def _ptrs(self):
        """ctypes pointer arrays of the current input and output tensors (rebuilt
        only when a tensor changes, to keep the per-launch host cost low)."""
        key = tuple(t.data_ptr() for t in self.ins) + (None,) + tuple(t.data_ptr() for t in self.outs)
        if getattr(self, "_ptr_key", None) != key:
            self._ptr_key = key
            self._ptr_arrays = (pointer_array([t.data_ptr() for t in self.ins]),
                                pointer_array([t.data_ptr() for t in self.outs]))
        return self._ptr_arrays

    def launch(self, stream=None):
        s = stream if stream is not None else torch.cuda.current_stream()
        ins, outs = self._ptrs()
        self.plan.execute(ins, outs, self.ws.data_ptr(), self.ws_bytes, s.cuda_stream)

    def launch_kernels(self, first, count, stream=None):
        s = stream if stream is not None else torch.cuda.current_stream()
        ins, outs = self._ptrs()
        self.plan.execute_kernels(first, count, ins, outs, self.ws.data_ptr(), self.ws_bytes, s.cuda_stream)

    def bind(self, stream=None):
        """Builds every C argument of one plan execution on ``stream`` (default:
        the current stream) once, for ``launch_bound`` / ``launch_timed_bound``:
        one library call per launch with no per-call conversions.  Bind again
        after ``set_inputs``."""
        s = stream if stream is not None else torch.cuda.current_stream()
        ins, outs = self._ptrs()
        self._bound = (self.plan.h, ins, outs, C.c_void_p(self.ws.data_ptr()), C.c_size_t(self.ws_bytes),
                       C.c_void_p(s.cuda_stream))
        self._nk = self.plan.num_kernels()
        return self

    def launch_bound(self):
        rc = lib.korch_plan_execute(*self._bound)
        if rc:
            check(rc)

    def event_arrays(self, starts, stops):
        """C arrays (one entry per kernel) of the hipEvent_t handles of torch
        events (each recorded once before, so that it exists) or None."""
        n = self._nk if hasattr(self, "_nk") else self.plan.num_kernels()
        a = (C.c_void_p * n)(*[e.cuda_event if e is not None else None for e in starts])
        b = (C.c_void_p * n)(*[e.cuda_event if e is not None else None for e in stops])
        return a, b

    def launch_events_bound(self, arrays):
        """One execution on the bound arguments with per-kernel dispatch events
        (``arrays`` from ``event_arrays``): korch_plan_execute_events."""
        h, ins, outs, ws, wsb, st = self._bound
        rc = lib.korch_plan_execute_events(h, ins, outs, ws, wsb, st, C.cast(arrays[0], C.POINTER(C.c_void_p)),
                                           C.cast(arrays[1], C.POINTER(C.c_void_p)))
        if rc:
            check(rc)

    def launch_timed_bound(self, timed, start, stop):
        """``launch_timed`` on the bound arguments (``start`` / ``stop``: torch events, each recorded once before)."""
        h, ins, outs, ws, wsb, st = self._bound
        rc = lib.korch_plan_execute_timed(h, 0, self._nk, ins, outs, ws, wsb, st, timed, C.c_void_p(start.cuda_event),
                                          C.c_void_p(stop.cuda_event))
        if rc:
            check(rc)

    def launch_timed(self, timed, start, stop, stream=None):
        """One execution of the whole plan with kernel ``timed`` bracketed by the
        torch events ``start`` / ``stop`` (each recorded once before, so that it exists)."""
        s = stream if stream is not None else torch.cuda.current_stream()
        ins, outs = self._ptrs()
        self.plan.execute_timed(0, self.plan.num_kernels(), ins, outs, self.ws.data_ptr(), self.ws_bytes,
                                s.cuda_stream, timed, start.cuda_event, stop.cuda_event)

    def run(self, storage: dict = None):
        if storage is not None:
            self.set_inputs(storage)
        self.launch()
        torch.cuda.synchronize()
        return {n: to_f64(t) for n, t in zip(self.w.output_names, self.outs)}
