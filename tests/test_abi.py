"""C-ABI library: loads, exports what include/dtr_sim.h declares, and
validates traces on the host (no GPU needed for any of these)."""
import ctypes as C
import re

import numpy as np
import pytest

from paper_2006_09616_amd import dtr as D
from paper_2006_09616_amd import workloads as W


def test_library_exports_every_declared_function():
    names = D.header_functions()
    assert set(names) >= {"dtr_sim_workspace_bytes", "dtr_sim_create", "dtr_sim_run",
                          "dtr_sim_results", "dtr_sim_destroy", "dtr_sim_last_error"}
    lib = D.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_spec_layout_matches_header():
    """Field offsets of the Python spec record against the C struct in the
    header (parsed, not restated)."""
    text = open(D.HEADER).read()
    body = text[text.index("typedef struct {", text.index("DTR_POLICY_BANISH")):text.index("} dtr_sim_spec;")]
    fields = [l.split()[-1].rstrip(";") for l in body.splitlines() if l.strip().endswith(";")]
    assert fields == list(W.SPEC_DTYPE.names)


def test_struct_sizes_match_header():
    assert C.sizeof(D._Trace) == 8 + 6 * 8
    assert W.SPEC_DTYPE.itemsize == 32
    assert D.RESULT_DTYPE.itemsize == 104


def test_launch_info_layout_and_null_arguments():
    text = open(D.HEADER).read()
    body = text[text.index("typedef struct {", text.index("dtr_sim_launch_info") - 900):text.index("} dtr_launch_info;")]
    fields = [l.split()[1].rstrip(";") for l in body.splitlines() if l.strip().startswith("int32_t")]
    assert fields == [f for f, _ in D._LaunchInfo._fields_]
    assert C.sizeof(D._LaunchInfo) == 16
    L = D.lib()
    assert L.dtr_sim_launch_info(None, None) == D.DTR_EINVAL


def _spec(h=W.H_LRU, b=10, trace=0):
    return W.make_specs([(trace, h, b, 0)])


def _expect(code, traces, specs, match):
    with pytest.raises(D.DtrError) as e:
        D.dtr_sim_workspace_bytes(traces, specs)
    assert e.value.code == code
    assert match in str(e.value)


def test_validation_rejects_malformed_traces():
    good = W.chain_trace(4)

    def mod(**kw):
        t = W.Trace("m", good.tensor_size.copy(), good.tensor_flags.copy(), good.op_output.copy(),
                    good.op_cost.copy(), good.op_input_offsets.copy(), good.op_inputs.copy())
        for k, v in kw.items():
            getattr(t, k)[...] = v
        return t

    t = mod()
    t.op_cost[2] = 0
    _expect(D.DTR_ETRACE, [t], _spec(), "op 2: cost 0")
    t = mod()
    t.tensor_size[1] = 0
    _expect(D.DTR_ETRACE, [t], _spec(), "tensor 1 size 0")
    t = mod()
    t.op_inputs[0] = 3                       # op 1 reads a tensor produced later
    _expect(D.DTR_ETRACE, [t], _spec(), "op 1: input 3 is not defined before use")
    t = mod()
    t.op_output[3] = 2                       # produced twice
    _expect(D.DTR_ETRACE, [t], _spec(), "already produced")
    t = mod()
    t.tensor_flags[0] = W.FLAG_CONSTANT      # constant that an op also produces
    _expect(D.DTR_ETRACE, [t], _spec(), "op 0: tensor 0 is a constant")
    t = mod()
    t.tensor_flags[2] = 8
    _expect(D.DTR_ETRACE, [t], _spec(), "unknown flag")
    _expect(D.DTR_ETRACE, [good], _spec(h=9), "unknown heuristic 9")
    for h in (8, 15, 32, -1):
        _expect(D.DTR_ETRACE, [good], _spec(h=h), f"unknown heuristic {h}")
    _expect(D.DTR_ETRACE, [good], W.make_specs([(0, W.H_LRU, 4, 0, 3)]), "unknown deallocation policy 3")
    _expect(D.DTR_ETRACE, [good], W.make_specs([(0, W.H_EQ, 4, 0, W.POLICY_BANISH)]),
            "banishing is not defined for union-find heuristics")
    _expect(D.DTR_ETRACE, [good], W.make_specs([(0, W.h_family(W.C_EQCLASS, 0, 1), 4, 0, W.POLICY_BANISH)]),
            "banishing is not defined for union-find heuristics")
    _expect(D.DTR_ETRACE, [good], W.make_specs([(0, W.H_LRU, 4, 0, 0, 4)]), "unknown search flags 4")
    _expect(D.DTR_ETRACE, [good], _spec(trace=1), "trace index 1 out of range")
    _expect(D.DTR_ETRACE, [good], _spec(b=-1), "negative budget")


def test_duplicate_input_rejected():
    ins = [[], [0], [0, 1, 1]]
    off = np.array([0, 0, 1, 4], np.int64)
    t = W.Trace("dup", np.ones(3, np.int64), np.zeros(3, np.uint8), np.arange(3, dtype=np.int32),
                np.ones(3, np.int64), off, np.array([0, 0, 1, 1], np.int32))
    _expect(D.DTR_ETRACE, [t], _spec(), "duplicate input 1")


def test_cost_sum_guard():
    n = 8
    t = W.Trace("big", np.ones(n, np.int64), np.zeros(n, np.uint8), np.arange(n, dtype=np.int32),
                np.full(n, 1 << 28, np.int64), np.zeros(n + 1, np.int64), np.zeros(0, np.int32))
    big = [t] * 1
    # 8 * 2^28 < 2^50: accepted by validation (may then fail only for lack of a GPU)
    try:
        D.dtr_sim_workspace_bytes(big, _spec())
    except D.DtrError as e:
        assert e.code == D.DTR_EHIP
    t2 = W.Trace("big", np.ones(n, np.int64), np.zeros(n, np.uint8), np.arange(n, dtype=np.int32),
                 np.full(n, (1 << 28) + 1, np.int64), np.zeros(n + 1, np.int64), np.zeros(0, np.int32))
    _expect(D.DTR_ETRACE, [t2], _spec(), "outside [1, 2^28]")


def test_null_arguments():
    lib = D.lib()
    assert lib.dtr_sim_workspace_bytes(None, 0, None, 0, None, None) == D.DTR_EINVAL
    assert lib.dtr_sim_run(None, None) == D.DTR_EINVAL
    assert lib.dtr_sim_results(None, None, 0) == D.DTR_EINVAL
    lib.dtr_sim_destroy(None)
    h = C.c_void_p()
    assert lib.dtr_sim_create(None, 0, None, 0, None, None, 0, None, C.byref(h)) == D.DTR_EINVAL
    assert "null" in D.dtr_sim_last_error()


def test_family_and_msps_ids_accepted():
    """Validation accepts h_MSPS and every family id (without a GPU the call
    then stops at the device query, after validation)."""
    good = W.chain_trace(4)
    for h in [W.H_MSPS] + W.ALL_FAMILY:
        try:
            assert D.dtr_sim_workspace_bytes([good], W.make_specs([(0, h, 4, 0)])) > 0
        except D.DtrError as e:
            assert e.code == D.DTR_EHIP and "heuristic" not in str(e), (h, str(e))


def test_log_struct_matches_header():
    text = open(D.HEADER).read()
    body = text[text.index("typedef struct {", text.index("DTR_LOG_RELEASE")):text.index("} dtr_log;")]
    fields = [l.split(";")[0].split()[-1].lstrip("*") for l in body.splitlines() if ";" in l]
    assert fields == [f for f, _ in D._Log._fields_]
    kinds = {k: int(v) for k, v in re.findall(r"#define DTR_LOG_(\w+)\s+(\d+)", text)}
    assert kinds == {n: getattr(W, "LOG_" + n) for n in kinds}


def _log_expect(logs, specs, match, code=None):
    with pytest.raises(D.DtrError) as e:
        D.dtr_log_workspace_bytes(logs, specs)
    assert e.value.code == (D.DTR_ETRACE if code is None else code), str(e.value)
    assert match in str(e.value), str(e.value)


def _rows(kind_rows):
    """A log from (kind, a, b, value, ins, outs) rows."""
    b = W.LogBuilder("m")
    for k, a_, b_, v, ins, outs in kind_rows:
        b._row(k, a_, b_, v, ins, outs)
    b.next_name = 1 + max([r[1] for r in kind_rows] + [x for r in kind_rows for x in r[4] + r[5]] + [0])
    return b.build()


def test_log_validation_rejects_malformed_logs():
    M, A, CALL, MUT, CONST, COPY, CF, REL = (W.LOG_MEMORY, W.LOG_ALIAS, W.LOG_CALL, W.LOG_MUTATE,
                                              W.LOG_CONSTANT, W.LOG_COPY, W.LOG_COPYFROM, W.LOG_RELEASE)
    sp = W.make_specs([(0, W.H_LRU, 10, 0)])
    good = [(CALL, -1, -1, 3, [], [0]), (M, 0, -1, 4, [], []), (A, 0, -1, 0, [], [])]
    cases = [
        ([(CALL, -1, -1, 3, [5], [0]), (M, 0, -1, 4, [], []), (A, 0, -1, 0, [], [])], "input name 5 is not bound"),
        (good + [(CALL, -1, -1, 3, [0], [0]), (M, 0, -1, 4, [], []), (A, 0, -1, 0, [], [])], "output name 0 is not fresh"),
        ([(CALL, -1, -1, 0, [], [0]), (M, 0, -1, 4, [], []), (A, 0, -1, 0, [], [])], "cost 0 outside"),
        ([(CALL, -1, -1, 3, [], [0]), (M, 0, -1, 0, [], []), (A, 0, -1, 0, [], [])], "size 0 outside"),
        ([(CALL, -1, -1, 3, [], [0]), (M, 0, -1, 4, [], [])], "outputs are not all described"),
        ([(CALL, -1, -1, 3, [], [0]), (A, 0, -1, 0, [], []), (M, 0, -1, 4, [], [])], "MEMORY then ALIAS"),
        ([(CALL, -1, -1, 3, [], [0]), (M, 0, -1, 4, [], []), (A, 0, 7, 0, [], [])], "neither an input"),
        ([(CALL, -1, -1, 3, [], []), ], "a call has no output"),
        (good + [(MUT, -1, -1, 2, [0], [3])], "mutated name 3 is not a distinct input"),
        (good + [(MUT, -1, -1, 2, [0], [0, 0])], "mutated name 0 is not a distinct input"),
        (good + [(REL, 0, -1, 0, [], []), (REL, 0, -1, 0, [], [])], "release of unbound name 0"),
        (good + [(COPY, 0, 0, 0, [], [])], "copy 0 <- 0"),
        (good + [(CF, 4, 0, 0, [], [])], "copyfrom 4 <- 0"),
        ([(CONST, 0, -1, 0, [], []), (M, 1, -1, 3, [], [])], "not followed by its MEMORY"),
        ([(M, 0, -1, 3, [], [])], "unexpected instruction kind 0"),
        ([(9, 0, -1, 3, [], [])], "unexpected instruction kind 9"),
    ]
    for rows, match in cases:
        _log_expect([_rows(rows)], sp, match)
    # two outputs of one call: the second views the first's new storage (accepted)
    ok = _rows([(CALL, -1, -1, 3, [], [0, 1]), (M, 0, -1, 4, [], []), (A, 0, -1, 0, [], []),
                (M, 1, -1, 4, [], []), (A, 1, 0, 0, [], [])])
    try:
        D.dtr_log_workspace_bytes([ok], sp)
    except D.DtrError as e:
        assert e.code == D.DTR_EHIP, str(e)
    _log_expect([ok], W.make_specs([(1, W.H_LRU, 10, 0)]), "log index 1 out of range")
    _log_expect([ok], W.make_specs([(0, W.H_EQ, 10, 0, W.POLICY_BANISH)]),
                "banishing is not defined for union-find heuristics")
    _log_expect([ok], W.make_specs([(0, 12, 10, 0)]), "unknown heuristic 12")


def test_generated_logs_pass_validation():
    """Every generator's logs are accepted (without a GPU the call then stops
    at the device query, after lowering)."""
    logs = [W.random_log(s, n_steps=80) for s in range(10)] + [W.log_from_trace(W.chain_trace(20))]
    specs = W.make_specs([(i, h, 50, 0) for i in range(len(logs)) for h in (W.H_DTR, W.H_EQ, W.H_MSPS)])
    try:
        assert D.dtr_log_workspace_bytes(logs, specs) > 0
    except D.DtrError as e:
        assert e.code == D.DTR_EHIP, str(e)


def test_log_options():
    """DTR_OPT_LOG_NO_LDS is accepted for logs only; other bits are rejected."""
    lib = D.lib()
    ok = W.log_from_trace(W.chain_trace(4))
    sp = W.make_specs([(0, W.H_DTR, 4, 0)])
    for flags, want in ((D.OPT_LOG_NO_LDS, None), (2, D.DTR_EINVAL)):
        try:
            D.dtr_log_workspace_bytes([ok], sp, {"slots": 0, "flags": flags})
            got = None
        except D.DtrError as e:
            got = e.code
        if want is None:
            assert got in (None, D.DTR_EHIP)
        else:
            assert got == want
    with pytest.raises(D.DtrError) as e:
        D.dtr_sim_workspace_bytes([W.chain_trace(4)], sp, {"slots": 0, "flags": D.OPT_LOG_NO_LDS})
    assert e.value.code == D.DTR_EINVAL


def test_static_scratch_option_limits():
    """DTR_OPT_STATIC_SCRATCH is for traces only, and a batch whose one
    simulation needs more working memory than the static array is rejected
    when the workspace is sized (before any device work)."""
    sp = W.make_specs([(0, W.H_DTR, 4, 0)])
    with pytest.raises(D.DtrError) as e:
        D.dtr_log_workspace_bytes([W.log_from_trace(W.chain_trace(4))], sp,
                                  {"slots": 0, "flags": D.OPT_STATIC_SCRATCH})
    assert e.value.code == D.DTR_EINVAL
    big = W.chain_trace(600_000)                   # 1.2M tensors: pool, remat stack and walk state > 256 MiB
    with pytest.raises(D.DtrError) as e:
        D.dtr_sim_workspace_bytes([big], sp, {"slots": 0, "flags": D.OPT_STATIC_SCRATCH})
    assert e.value.code == D.DTR_EINVAL and "static scratch" in str(e.value)


def test_progress_null_arguments():
    """dtr_sim_progress rejects a NULL handle or output without device work."""
    L = D.lib()
    v = C.c_int64(7)
    assert L.dtr_sim_progress(None, C.byref(v)) == D.DTR_EINVAL
    assert L.dtr_sim_progress(None, None) == D.DTR_EINVAL
