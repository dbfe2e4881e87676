"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: a
stand-alone driver (tests/oracle_sanitize_main.c, which includes the oracle's
source) is built with both sanitizers and replays random programs, chains,
the clock-overflow cases and random operator logs under every heuristic,
deallocation policy and search flag; it must report no error and return the
results the ordinary build returns."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2006_09616_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _write(path, traces, specs, logs, lspecs):
    i32 = lambda v: np.asarray([v], "<i4").tobytes()
    with open(path, "wb") as f:
        f.write(i32(len(traces)))
        for t in traces:
            f.write(i32(t.n_tensors) + i32(t.n_ops))
            for a, dt in ((t.tensor_size, "<i8"), (t.tensor_flags, "u1"), (t.op_output, "<i4"),
                          (t.op_cost, "<i8"), (t.op_input_offsets, "<i8"), (t.op_inputs, "<i4")):
                f.write(np.ascontiguousarray(a, dt).tobytes())
        f.write(i32(len(specs)) + np.ascontiguousarray(specs, W.SPEC_DTYPE).tobytes())
        f.write(i32(len(logs)))
        for g in logs:
            f.write(i32(int(g.n_instrs)) + i32(int(g.n_names)))
            for a, dt in ((g.kind, "<i4"), (g.a, "<i4"), (g.b, "<i4"), (g.n_in, "<i4"), (g.value, "<i8"),
                          (g.list_offsets, "<i8"), (g.ids, "<i4")):
                f.write(np.ascontiguousarray(a, dt).tobytes())
        f.write(i32(len(lspecs)) + np.ascontiguousarray(lspecs, W.SPEC_DTYPE).tobytes())


def _inputs():
    traces, rows = [], []
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS,
          W.h_family(W.C_ESTAR, 0, 0), W.h_family(W.C_EQCLASS, 1, 0)]
    uf = {W.H_EQ, W.h_family(W.C_EQCLASS, 1, 0)}
    for s in range(24):
        tr = W.random_program(3100 + s, n_ops=8 + (s * 7) % 60, n_const=s % 3, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + s % 12, max_cost=1 + s % 6)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for h in hs:
            for pol in (W.POLICY_EAGER, W.POLICY_IGNORE, W.POLICY_BANISH):
                if pol == W.POLICY_BANISH and h in uf:
                    continue
                for frac in (0.3, 0.7):
                    rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s, pol, s % 4))
    traces.append(W.chain_trace(40))
    traces.append(W.shared_weight_chain(300))
    for i in (len(traces) - 2, len(traces) - 1):
        for h in hs:
            rows.append((i, h, 6, 1))
    traces.append(W.plain_chain(4096, 1 << 28, True, [-1]))
    for h in hs:
        rows.append((len(traces) - 1, h, 2, 1))
    logs = [W.random_log(s, n_steps=50, n_const=2) for s in range(10)]
    lrows = [(i, h, max(1, W.log_peak(logs[i]) // d), 7 + i, pol)
             for i in range(len(logs)) for h in (W.H_DTR, W.H_EQ, W.H_LRU, W.H_MSPS) for d in (2, 3)
             for pol in (W.POLICY_EAGER, W.POLICY_BANISH) if not (h == W.H_EQ and pol == W.POLICY_BANISH)]
    return traces, W.make_specs(rows), logs, W.make_specs(lrows)


def test_oracle_under_sanitizers(oracle_lib, tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("no gcc")
    exe = tmp_path / "oracle_sanitize"
    build = subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer",
                            "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-pthread",
                            "-o", str(exe), os.path.join(HERE, "oracle_sanitize_main.c")],
                           capture_output=True, text=True)
    if build.returncode != 0 and "asan" in build.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + build.stderr[-300:])
    assert build.returncode == 0, build.stderr
    traces, specs, logs, lspecs = _inputs()
    inp, out = tmp_path / "in.bin", tmp_path / "out.bin"
    _write(inp, traces, specs, logs, lspecs)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    run = subprocess.run([str(exe), str(inp), str(out), "4"], capture_output=True, text=True, env=env,
                         timeout=600)
    assert run.returncode == 0, run.stderr[-3000:]
    assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr, run.stderr[-3000:]
    nf = len(oracle_lib.RESULT_FIELDS)
    got = np.fromfile(out, "<i8").reshape(-1, nf)
    assert got.shape[0] == len(specs) + len(lspecs)
    ref = oracle_lib.run(traces, specs)
    lref = oracle_lib.run_log(logs, lspecs)
    want = np.concatenate([np.stack([ref[f] for f in oracle_lib.RESULT_FIELDS], 1),
                           np.stack([lref[f] for f in oracle_lib.RESULT_FIELDS], 1)])
    assert (got == want).all()
    assert (ref["status"] == oracle_lib.STATUS_CLOCK_OVERFLOW).any() and (ref["status"] == oracle_lib.STATUS_OOM).any()


def _malformed():
    """Traces and logs the host must reject, one per input file."""
    base = W.random_program(7, n_ops=20, n_const=2, backward=True)
    out = []
    t = W.Trace("oob", base.tensor_size, base.tensor_flags, base.op_output, base.op_cost,
                base.op_input_offsets, base.op_inputs.copy())
    t.op_inputs[3] = base.n_tensors + 5                      # input out of range
    out.append(t)
    t = W.Trace("dup", base.tensor_size, base.tensor_flags, base.op_output, base.op_cost,
                base.op_input_offsets, base.op_inputs.copy())
    o = int(np.argmax(np.diff(base.op_input_offsets) >= 2))
    b = int(base.op_input_offsets[o])
    t.op_inputs[b + 1] = t.op_inputs[b]                      # duplicate input
    out.append(t)
    sz = base.tensor_size.copy()
    sz[0] = 1 << 36                                          # size at the limit
    out.append(W.Trace("size", sz, base.tensor_flags, base.op_output, base.op_cost, base.op_input_offsets,
                       base.op_inputs))
    cost = base.op_cost.copy()
    cost[1] = 0                                              # cost below 1
    out.append(W.Trace("cost", base.tensor_size, base.tensor_flags, base.op_output, cost,
                       base.op_input_offsets, base.op_inputs))
    off = base.op_input_offsets.copy()
    off[2], off[3] = off[3], off[2]                          # offsets not monotone
    out.append(W.Trace("off", base.tensor_size, base.tensor_flags, base.op_output, base.op_cost, off,
                       base.op_inputs))
    return out


def test_host_code_under_sanitizers(tmp_path):
    """Validation, derivation, log lowering and workspace layout under
    AddressSanitizer and UndefinedBehaviorSanitizer: valid batches get as far
    as the device query (DTR_EHIP here), malformed traces are rejected."""
    gxx = shutil.which("g++")
    hip_inc, hip_lib = "/opt/rocm/include", "/opt/rocm/lib"
    if not gxx or not os.path.isdir(hip_inc):
        pytest.skip("no g++ or HIP headers")
    exe = tmp_path / "host_sanitize"
    csrc = os.path.join(ROOT, "paper_2006_09616_amd", "csrc")
    build = subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
                            "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                            "-D__HIP_PLATFORM_AMD__", "-I", hip_inc, "-I", os.path.join(ROOT, "include"),
                            "-o", str(exe), os.path.join(HERE, "host_sanitize_main.cpp"),
                            os.path.join(csrc, "dtr_sim.cpp"), os.path.join(csrc, "dtr_log.cpp"),
                            "-L", hip_lib, "-Wl,-rpath," + hip_lib, "-lamdhip64"],
                           capture_output=True, text=True)
    if build.returncode != 0 and ("asan" in build.stderr.lower() or "amdhip64" in build.stderr):
        pytest.skip("sanitizer runtime or HIP library not available: " + build.stderr[-300:])
    assert build.returncode == 0, build.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:exitcode=23",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1:exitcode=24")
    traces, specs, logs, lspecs = _inputs()
    cases = [(traces, specs, logs, lspecs, {0, -3})]
    for t in _malformed():
        cases.append(([t], W.make_specs([(0, W.H_DTR, 10, 0)]), [], W.make_specs([]), {-2, -1}))
    for k, (tr, sp, lg, lsp, ok) in enumerate(cases):
        inp = tmp_path / f"in{k}.bin"
        _write(inp, tr, sp, lg, lsp)
        run = subprocess.run([str(exe), str(inp)], capture_output=True, text=True, env=env, timeout=300)
        assert run.returncode == 0, run.stderr[-3000:]
        assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr, run.stderr[-3000:]
        rc = [int(v) for v in run.stdout.split()]
        assert rc[0] in ok, (k, rc)
        if k == 0:
            assert rc[1] in ok, (k, rc)
