"""ctypes front end of the CPU oracle (``dtr_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, by the smoke check and
by the benchmark's CPU-baseline leg, never by the GPU path.  The oracle is a
plain step-by-step rendering of the DTR greedy loop (Section 2, Appendix C);
see the header of ``dtr_oracle.c`` for what it follows and which readings it
takes where the paper is silent.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "dtr_oracle.c")
LIB = os.path.join(HERE, "libdtr_oracle.so")

RESULT_FIELDS = ["total_cost", "base_cost", "remat_cost", "peak_memory", "final_memory",
                 "n_executed_ops", "n_remats", "n_evictions", "n_eager_evictions", "n_scores",
                 "n_nbr_visits", "n_adj_visits", "status", "failed_op"]
RESULT_DTYPE = np.dtype([(f, "<i8") for f in RESULT_FIELDS])

STATUS_OK, STATUS_OOM, STATUS_CLOCK_OVERFLOW, STATUS_STOPPED = 0, 1, 2, 100
UNCOMPUTED, RESIDENT, EVICTED, BANISHED = 0, 1, 2, 3


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C11, pthreads).

    ``DTR_ORACLE_LIB`` names another build of the same interface to load
    instead (the mutation test runs the pins against deliberately broken
    copies of the source this way)."""
    other = os.environ.get("DTR_ORACLE_LIB")
    if other:
        return other
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-pthread", "-o", tmp, SRC])
        os.replace(tmp, LIB)
    return LIB


class _Trace(C.Structure):
    _fields_ = [("n_tensors", C.c_int32), ("n_ops", C.c_int32),
                ("tensor_size", C.c_void_p), ("tensor_flags", C.c_void_p),
                ("op_output", C.c_void_p), ("op_cost", C.c_void_p),
                ("op_input_offsets", C.c_void_p), ("op_inputs", C.c_void_p)]


class _Probe(C.Structure):
    _fields_ = [("stop_after_op", C.c_int64), ("stop_at_eviction", C.c_int64),
                ("state_out", C.c_void_p), ("locks_out", C.c_void_p), ("last_out", C.c_void_p),
                ("score_n_out", C.c_void_p), ("score_d_lo_out", C.c_void_p),
                ("score_d_hi_out", C.c_void_p), ("candidate_out", C.c_void_p),
                ("clock_out", C.c_void_p),
                ("evict_log", C.c_void_p), ("evict_log_cap", C.c_int64), ("evict_log_len", C.c_void_p),
                ("remat_log", C.c_void_p), ("remat_log_cap", C.c_int64), ("remat_log_len", C.c_void_p),
                ("uf_cost_sum_out", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        _lib.oracle_run.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p,
                                    C.c_int32, C.c_void_p]
        _lib.oracle_run.restype = C.c_int
        _lib.oracle_result_fields.restype = C.c_int
        _lib.oracle_estar.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int32]
        _lib.oracle_estar.restype = C.c_int64
        _lib.oracle_rand_key.argtypes = [C.c_uint64, C.c_int64, C.c_int32]
        _lib.oracle_rand_key.restype = C.c_uint64
        _lib.oracle_sample_key.argtypes = [C.c_uint64, C.c_int64, C.c_int32]
        _lib.oracle_sample_key.restype = C.c_uint64
        assert _lib.oracle_result_fields() == len(RESULT_FIELDS)
    return _lib


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def _pack(traces):
    arr = (_Trace * max(1, len(traces)))()
    keep = []
    for i, t in enumerate(traces):
        cols = [np.ascontiguousarray(t.tensor_size, np.int64), np.ascontiguousarray(t.tensor_flags, np.uint8),
                np.ascontiguousarray(t.op_output, np.int32), np.ascontiguousarray(t.op_cost, np.int64),
                np.ascontiguousarray(t.op_input_offsets, np.int64), np.ascontiguousarray(t.op_inputs, np.int32)]
        keep.extend(cols)
        arr[i] = _Trace(t.n_tensors, t.n_ops, *[c.ctypes.data for c in cols])
    return arr, keep


def run(traces, specs, threads: int | None = None) -> np.ndarray:
    """Run every simulation in ``specs`` (SPEC_DTYPE array) and return a
    RESULT_DTYPE array, one row per simulation."""
    specs = np.ascontiguousarray(specs)
    arr, keep = _pack(traces)
    out = np.zeros(len(specs), dtype=RESULT_DTYPE)
    threads = threads or os.cpu_count() or 1
    rc = lib().oracle_run(C.addressof(arr), len(traces), _ptr(specs), len(specs), _ptr(out),
                          int(threads), None)
    if rc != 0:
        raise RuntimeError(f"oracle_run failed with {rc}")
    del keep
    return out


class _Log(C.Structure):
    _fields_ = [("n_instrs", C.c_int32), ("n_names", C.c_int32), ("kind", C.c_void_p), ("a", C.c_void_p),
                ("b", C.c_void_p), ("n_in", C.c_void_p), ("value", C.c_void_p), ("list_offsets", C.c_void_p),
                ("ids", C.c_void_p)]


def run_log(logs, specs, threads: int | None = None) -> np.ndarray:
    """Replay operator logs (the spec's trace field indexes ``logs``); one
    RESULT_DTYPE row per simulation."""
    specs = np.ascontiguousarray(specs)
    arr = (_Log * max(1, len(logs)))()
    keep = []
    for i, g in enumerate(logs):
        cols = [np.ascontiguousarray(g.kind, np.int32), np.ascontiguousarray(g.a, np.int32),
                np.ascontiguousarray(g.b, np.int32), np.ascontiguousarray(g.n_in, np.int32),
                np.ascontiguousarray(g.value, np.int64), np.ascontiguousarray(g.list_offsets, np.int64),
                np.ascontiguousarray(g.ids, np.int32)]
        keep.extend(cols)
        arr[i] = _Log(g.n_instrs, g.n_names, *[c.ctypes.data for c in cols])
    out = np.zeros(len(specs), dtype=RESULT_DTYPE)
    threads = threads or os.cpu_count() or 1
    L = lib()
    L.oracle_run_log.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32]
    L.oracle_run_log.restype = C.c_int
    rc = L.oracle_run_log(C.addressof(arr), len(logs), _ptr(specs), len(specs), _ptr(out), int(threads))
    del keep
    if rc != 0:
        raise RuntimeError(f"oracle_run_log failed with {rc}")
    return out


def run_probe(trace, spec, stop_after_op: int = -1, stop_at_eviction: int = -1,
              log_cap: int = 1 << 20) -> dict:
    """One simulation with the test probes: state at a stop point, every
    candidate's score at a given budget-eviction decision, and the logs of
    evicted and rematerialized tensor ids."""
    n = trace.n_tensors
    state = np.zeros(n, np.uint8)
    locks = np.zeros(n, np.int32)
    last = np.zeros(n, np.int64)
    sn = np.zeros(n, np.uint64)
    sdl = np.zeros(n, np.uint64)
    sdh = np.zeros(n, np.uint64)
    cand = np.zeros(n, np.uint8)
    clock = np.zeros(1, np.int64)
    elog = np.zeros(log_cap, np.int32)
    elen = np.zeros(1, np.int64)
    rlog = np.zeros(log_cap, np.int32)
    rlen = np.zeros(1, np.int64)
    ufsum = np.zeros(1, np.int64)
    pr = _Probe(stop_after_op, stop_at_eviction, state.ctypes.data, locks.ctypes.data,
                last.ctypes.data, sn.ctypes.data, sdl.ctypes.data, sdh.ctypes.data,
                cand.ctypes.data, clock.ctypes.data, elog.ctypes.data, log_cap, elen.ctypes.data,
                rlog.ctypes.data, log_cap, rlen.ctypes.data, ufsum.ctypes.data)
    specs = np.ascontiguousarray(np.asarray([spec]).reshape(1))
    arr, keep = _pack([trace])
    out = np.zeros(1, dtype=RESULT_DTYPE)
    specs = specs.copy()
    specs["trace"] = 0
    rc = lib().oracle_run(C.addressof(arr), 1, _ptr(specs), 1, _ptr(out), 1, C.addressof(pr))
    if rc != 0:
        raise RuntimeError(f"oracle_run failed with {rc}")
    del keep
    D = [int(lo) | (int(hi) << 64) for lo, hi in zip(sdl.tolist(), sdh.tolist())]
    return dict(result=out[0], state=state, locks=locks, last_access=last, clock=int(clock[0]),
                score_n=[int(v) for v in sn.tolist()], score_d=D, candidate=cand.astype(bool),
                evict_log=elog[:elen[0]].copy(), remat_log=rlog[:rlen[0]].copy(),
                uf_cost_sum=int(ufsum[0]))


def estar(trace, state, x: int, ancestors_only: bool = False):
    """Exact evicted neighbourhood e*(x) under ``state`` (or e_R(x), the
    evicted ancestors only): (cost sum, members)."""
    arr, keep = _pack([trace])
    state = np.ascontiguousarray(state, np.uint8)
    cnt = np.zeros(1, np.int64)
    member = np.zeros(trace.n_tensors, np.uint8)
    s = lib().oracle_estar(C.addressof(arr), _ptr(state), int(x), _ptr(cnt), _ptr(member), int(ancestors_only))
    del keep
    if s < 0:
        raise RuntimeError("oracle_estar failed")
    return int(s), member.astype(bool)


def rand_key(seed: int, eviction_no: int, x: int) -> int:
    return int(lib().oracle_rand_key(seed, eviction_no, x))


def sample_key(seed: int, eviction_no: int, x: int) -> int:
    return int(lib().oracle_sample_key(seed, eviction_no, x))
