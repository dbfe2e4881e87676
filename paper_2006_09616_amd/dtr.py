"""Python binding of the C ABI in include/dtr_sim.h (argument marshalling only).

Every step of the simulation runs in the HIP library ``libdtrsim.so`` built
from ``csrc/``; this module only packs numpy arrays into the C structs, and
uses PyTorch for device memory (the workspace) and streams.  There is no
fallback: if the library is missing the calls raise.
"""
from __future__ import annotations

import ctypes as C
import os
import re

import numpy as np

from .workloads import SPEC_DTYPE

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdtrsim.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "dtr_sim.h")

DTR_OK, DTR_EINVAL, DTR_ETRACE, DTR_EHIP, DTR_ESTATE = 0, -1, -2, -3, -4
STATUS_OK, STATUS_OOM, STATUS_CLOCK_OVERFLOW, STATUS_CAPACITY = 0, 1, 2, 3
OPT_LOG_NO_LDS = 1
OPT_STATIC_SCRATCH = 2
OPT_WALK_QUEUE_SMALL = 4


def opt_walk_waves(w: int) -> int:
    """Option bits: w wavefronts per workgroup of the walk heuristics."""
    return w << 8

RESULT_FIELDS = ["total_cost", "base_cost", "remat_cost", "peak_memory", "final_memory",
                 "n_executed_ops", "n_remats", "n_evictions", "n_eager_evictions", "n_scores",
                 "n_nbr_visits", "n_adj_visits"]
RESULT_DTYPE = np.dtype([(f, "<i8") for f in RESULT_FIELDS] + [("status", "<i4"), ("failed_op", "<i4")])
assert RESULT_DTYPE.itemsize == 104


class DtrError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"dtr_sim error {code}: {message}")
        self.code = code


class _Trace(C.Structure):
    _fields_ = [("n_tensors", C.c_int32), ("n_ops", C.c_int32),
                ("tensor_size", C.c_void_p), ("tensor_flags", C.c_void_p),
                ("op_output", C.c_void_p), ("op_cost", C.c_void_p),
                ("op_input_offsets", C.c_void_p), ("op_inputs", C.c_void_p)]


class _Options(C.Structure):
    _fields_ = [("slots", C.c_int32), ("flags", C.c_int32)]


_lib = None


def lib():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        L.dtr_sim_workspace_bytes.argtypes = [vp, i32, vp, i32, vp, C.POINTER(sz)]
        L.dtr_sim_create.argtypes = [vp, i32, vp, i32, vp, vp, sz, vp, C.POINTER(vp)]
        L.dtr_sim_run.argtypes = [vp, vp]
        L.dtr_sim_run_static.argtypes = [vp, vp]
        L.dtr_sim_results.argtypes = [vp, vp, i32]
        L.dtr_sim_progress.argtypes = [vp, C.POINTER(C.c_int64)]
        L.dtr_sim_launch_info.argtypes = [vp, vp]
        L.dtr_sim_destroy.argtypes = [vp]
        L.dtr_sim_destroy.restype = None
        L.dtr_sim_last_error.restype = C.c_char_p
        L.dtr_log_workspace_bytes.argtypes = [vp, i32, vp, i32, vp, C.POINTER(sz)]
        L.dtr_log_create.argtypes = [vp, i32, vp, i32, vp, vp, sz, vp, C.POINTER(vp)]
        for f in ("dtr_sim_workspace_bytes", "dtr_sim_create", "dtr_sim_run", "dtr_sim_run_static", "dtr_sim_results",
                  "dtr_sim_progress", "dtr_sim_launch_info", "dtr_log_workspace_bytes", "dtr_log_create"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def header_functions():
    """Names of the functions declared in include/dtr_sim.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char \*)\s*\*?\s*(dtr_\w+)\s*\(", text, re.M)))


def dtr_sim_last_error() -> str:
    return lib().dtr_sim_last_error().decode()


def _check(rc: int):
    if rc != DTR_OK:
        raise DtrError(rc, dtr_sim_last_error())


class _Packed:
    """Keeps the numpy columns alive while the C structs point at them."""

    def __init__(self, traces, specs, options):
        self.cols = []
        self.arr = (_Trace * max(1, len(traces)))()
        for i, t in enumerate(traces):
            cols = [np.ascontiguousarray(t.tensor_size, np.int64), np.ascontiguousarray(t.tensor_flags, np.uint8),
                    np.ascontiguousarray(t.op_output, np.int32), np.ascontiguousarray(t.op_cost, np.int64),
                    np.ascontiguousarray(t.op_input_offsets, np.int64), np.ascontiguousarray(t.op_inputs, np.int32)]
            self.cols.extend(cols)
            self.arr[i] = _Trace(t.n_tensors, t.n_ops, *[c.ctypes.data for c in cols])
        self.n_traces = len(traces)
        self.specs = np.ascontiguousarray(specs, dtype=SPEC_DTYPE)
        self.opt = _Options(int(options.get("slots", 0)), int(options.get("flags", 0))) if options else None

    def args(self):
        return (C.addressof(self.arr), self.n_traces, self.specs.ctypes.data, len(self.specs),
                C.addressof(self.opt) if self.opt is not None else None)


class _Log(C.Structure):
    _fields_ = [("n_instrs", C.c_int32), ("n_names", C.c_int32), ("kind", C.c_void_p), ("a", C.c_void_p),
                ("b", C.c_void_p), ("n_in", C.c_void_p), ("value", C.c_void_p), ("list_offsets", C.c_void_p),
                ("ids", C.c_void_p)]


class _PackedLogs(_Packed):
    """Operator logs (``workloads.Log``) packed into ``dtr_log`` structs."""

    def __init__(self, logs, specs, options):
        self.cols = []
        self.arr = (_Log * max(1, len(logs)))()
        for i, g in enumerate(logs):
            cols = [np.ascontiguousarray(g.kind, np.int32), np.ascontiguousarray(g.a, np.int32),
                    np.ascontiguousarray(g.b, np.int32), np.ascontiguousarray(g.n_in, np.int32),
                    np.ascontiguousarray(g.value, np.int64), np.ascontiguousarray(g.list_offsets, np.int64),
                    np.ascontiguousarray(g.ids, np.int32)]
            self.cols.extend(cols)
            self.arr[i] = _Log(int(g.n_instrs), int(g.n_names), *[c.ctypes.data for c in cols])
        self.n_traces = len(logs)
        self.specs = np.ascontiguousarray(specs, dtype=SPEC_DTYPE)
        self.opt = _Options(int(options.get("slots", 0)), int(options.get("flags", 0))) if options else None


def dtr_log_workspace_bytes(logs, specs, options: dict | None = None) -> int:
    p = _PackedLogs(logs, specs, options)
    out = C.c_size_t(0)
    _check(lib().dtr_log_workspace_bytes(*p.args(), C.byref(out)))
    return int(out.value)


def dtr_log_create(logs, specs, workspace_ptr: int, workspace_bytes: int, stream_ptr: int,
                   options: dict | None = None) -> int:
    p = _PackedLogs(logs, specs, options)
    h = C.c_void_p()
    _check(lib().dtr_log_create(*p.args(), C.c_void_p(workspace_ptr), C.c_size_t(workspace_bytes),
                                C.c_void_p(stream_ptr), C.byref(h)))
    return int(h.value)


def dtr_sim_workspace_bytes(traces, specs, options: dict | None = None) -> int:
    p = _Packed(traces, specs, options)
    out = C.c_size_t(0)
    _check(lib().dtr_sim_workspace_bytes(*p.args(), C.byref(out)))
    return int(out.value)


def dtr_sim_create(traces, specs, workspace_ptr: int, workspace_bytes: int, stream_ptr: int,
                   options: dict | None = None) -> int:
    p = _Packed(traces, specs, options)
    h = C.c_void_p()
    _check(lib().dtr_sim_create(*p.args(), C.c_void_p(workspace_ptr), C.c_size_t(workspace_bytes),
                                C.c_void_p(stream_ptr), C.byref(h)))
    return int(h.value)


def dtr_sim_run(handle: int, stream_ptr: int):
    _check(lib().dtr_sim_run(C.c_void_p(handle), C.c_void_p(stream_ptr)))


def dtr_sim_run_static(handle: int, stream_ptr: int):
    _check(lib().dtr_sim_run_static(C.c_void_p(handle), C.c_void_p(stream_ptr)))


def dtr_sim_results(handle: int, n_sims: int) -> np.ndarray:
    out = np.zeros(n_sims, dtype=RESULT_DTYPE)
    _check(lib().dtr_sim_results(C.c_void_p(handle), out.ctypes.data, n_sims))
    return out


def dtr_sim_progress(handle: int) -> int:
    v = C.c_int64(0)
    _check(lib().dtr_sim_progress(C.c_void_p(handle), C.byref(v)))
    return int(v.value)


class _LaunchInfo(C.Structure):
    _fields_ = [("n_slots", C.c_int32), ("waves_per_group", C.c_int32), ("lds_bytes", C.c_int32),
                ("reserved", C.c_int32)]


def dtr_sim_launch_info(handle: int) -> dict:
    out = _LaunchInfo()
    _check(lib().dtr_sim_launch_info(C.c_void_p(handle), C.byref(out)))
    return {"n_slots": out.n_slots, "waves_per_group": out.waves_per_group, "lds_bytes": out.lds_bytes}


def dtr_sim_destroy(handle: int):
    if handle:
        lib().dtr_sim_destroy(C.c_void_p(handle))


class Simulator:
    """A batch on one GPU: workspace allocated as a torch uint8 tensor, work
    enqueued on a torch stream.  ``run()`` is asynchronous; ``results()``
    synchronizes."""

    def __init__(self, traces, specs, device: str = "cuda", slots: int = 0, stream=None, logs=None, flags: int = 0):
        """Simulate ``traces`` (dtr_trace), or operator ``logs`` (dtr_log)
        when given; the specs' trace field indexes whichever is given."""
        import torch
        lib()                                   # fail loudly before touching the GPU
        self.torch = torch
        self.device = torch.device(device)
        self.n_sims = len(specs)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        opts = {"slots": slots, "flags": flags} if (slots or flags) else None
        with torch.cuda.device(self.device):
            if logs is not None:
                self.bytes = dtr_log_workspace_bytes(logs, specs, opts)
                self.workspace = torch.empty(self.bytes, dtype=torch.uint8, device=self.device)
                self.handle = dtr_log_create(logs, specs, self.workspace.data_ptr(), self.bytes,
                                             self.stream.cuda_stream, opts)
            else:
                self.bytes = dtr_sim_workspace_bytes(traces, specs, opts)
                self.workspace = torch.empty(self.bytes, dtype=torch.uint8, device=self.device)
                self.handle = dtr_sim_create(traces, specs, self.workspace.data_ptr(), self.bytes,
                                             self.stream.cuda_stream, opts)

    def run(self):
        with self.torch.cuda.device(self.device):
            dtr_sim_run(self.handle, self.stream.cuda_stream)

    def run_static(self):
        """Run with the library's static working memory (dtr_sim_run_static)."""
        with self.torch.cuda.device(self.device):
            dtr_sim_run_static(self.handle, self.stream.cuda_stream)

    def results(self) -> np.ndarray:
        with self.torch.cuda.device(self.device):
            return dtr_sim_results(self.handle, self.n_sims)

    def progress(self) -> int:
        """Operations executed so far by the last run's walk-heuristic
        simulations, in steps of 4096 each (dtr_sim_progress; no wait)."""
        with self.torch.cuda.device(self.device):
            return dtr_sim_progress(self.handle)

    def done(self) -> bool:
        """Whether the work enqueued on the handle's stream has finished."""
        return bool(self.stream.query())

    def launch_info(self) -> dict:
        """Resident slots, waves per workgroup and dynamic LDS bytes."""
        return dtr_sim_launch_info(self.handle)

    def close(self):
        if getattr(self, "handle", 0):
            dtr_sim_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def run(traces, specs, device: str = "cuda", slots: int = 0, flags: int = 0) -> np.ndarray:
    """Simulate every spec on the GPU and return the results (numpy)."""
    sim = Simulator(traces, specs, device=device, slots=slots, flags=flags)
    try:
        sim.run()
        return sim.results()
    finally:
        sim.close()


def run_log(logs, specs, device: str = "cuda", slots: int = 0, flags: int = 0) -> np.ndarray:
    """Replay operator logs on the GPU (the specs' trace field indexes
    ``logs``) and return the results (numpy)."""
    sim = Simulator(None, specs, device=device, slots=slots, logs=logs, flags=flags)
    try:
        sim.run()
        return sim.results()
    finally:
        sim.close()
