"""GPU parity of operator-log replay (Appendix C.6): the HIP path, called
through the C ABI (dtr_log_create), against the CPU oracle's log replay,
field by field and bit-exact."""
import numpy as np
import pytest

import brute_log

from paper_2006_09616_amd import workloads as W

pytestmark = pytest.mark.gpu

FIELDS = ["total_cost", "base_cost", "remat_cost", "peak_memory", "final_memory", "n_executed_ops",
          "n_remats", "n_evictions", "n_eager_evictions", "n_scores", "n_nbr_visits", "n_adj_visits",
          "status", "failed_op"]
UF = {W.H_EQ} | {W.h_family(W.C_EQCLASS, s, m) for s in (0, 1) for m in (0, 1)}
HS = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS,
      W.h_family(W.C_ESTAR, 1, 0), W.h_family(W.C_EQCLASS, 0, 1), W.h_family(W.C_LOCAL, 1, 1),
      W.h_family(W.C_NONE, 0, 0)]


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2006_09616_amd import dtr as D
    D.lib()
    return D


def compare(got, ref, specs, label):
    bad = []
    for k in range(len(specs)):
        for f in FIELDS:
            if int(got[f][k]) != int(ref[f][k]):
                bad.append((k, f, int(got[f][k]), int(ref[f][k]), tuple(specs[k])))
                break
    assert not bad, f"{label}: {len(bad)}/{len(specs)} differ; first: {bad[:4]}"


def unlimited_peaks(O, logs):
    specs = W.make_specs([(i, W.H_LRU, W.BUDGET_UNLIMITED, 0) for i in range(len(logs))])
    return [int(v) for v in O.run_log(logs, specs)["peak_memory"]]


def rows_for(i, peak, seed, hs, policies=(W.POLICY_EAGER,), searches=(0,), fracs=(0.3, 0.6, 1.0)):
    rows = []
    for policy in policies:
        for search in searches:
            for h in hs:
                if policy == W.POLICY_BANISH and h in UF:
                    continue
                for frac in fracs:
                    rows.append((i, h, max(1, int(peak * frac)), seed * 97 + h, policy, search))
    return rows


@pytest.mark.parametrize("flags", [0, 1], ids=["lds", "device-memory"])
def test_random_logs_all_heuristics_and_policies(gpu, oracle_lib, flags):
    """Both kernel variants: walk state in LDS, and all in device memory."""
    logs = [W.random_log(s, n_steps=10 + (s * 13) % 140, n_const=s % 4, max_size=1 + s % 12,
                         max_cost=1 + s % 6, max_in=1 + s % 4, keep=s % 4) for s in range(48)]
    peaks = unlimited_peaks(oracle_lib, logs)
    rows = []
    for i, pk in enumerate(peaks):
        rows += rows_for(i, pk, i, HS, policies=(W.POLICY_EAGER, W.POLICY_IGNORE, W.POLICY_BANISH))
    specs = W.make_specs(rows)
    print(f"random logs: {len(logs)} logs, {len(specs)} sims, flags {flags}", flush=True)
    compare(gpu.run_log(logs, specs, flags=flags), oracle_lib.run_log(logs, specs), specs, "random logs")


def test_random_logs_search_approximations(gpu, oracle_lib):
    logs = [W.random_log(700 + s, n_steps=60 + (s * 29) % 200, n_const=s % 3, max_size=1 + (s * 7) % 60,
                         max_cost=1 + s % 5, max_in=1 + s % 4) for s in range(24)]
    peaks = unlimited_peaks(oracle_lib, logs)
    rows = []
    flags = (W.SEARCH_IGNORE_SMALL, W.SEARCH_SAMPLE, W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE)
    for i, pk in enumerate(peaks):
        rows += rows_for(i, pk, i, [W.H_DTR, W.H_EQ, W.H_LRU, W.H_RAND, W.H_MSPS], searches=flags,
                         fracs=(0.3, 0.6))
    specs = W.make_specs(rows)
    print(f"search logs: {len(specs)} sims", flush=True)
    compare(gpu.run_log(logs, specs), oracle_lib.run_log(logs, specs), specs, "search logs")


def test_plain_programs_as_logs(gpu, oracle_lib):
    """Traces written as logs (one storage per tensor), constants included."""
    logs = []
    rows = []
    for s in range(24):
        tr = W.random_program(300 + s, n_ops=15 + (s * 11) % 90, n_const=s % 3, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + s % 15, max_cost=1 + s % 6)
        logs.append(W.log_from_trace(tr))
        rows += rows_for(len(logs) - 1, W.natural_peak(tr), s, HS, policies=(W.POLICY_EAGER, W.POLICY_BANISH),
                         fracs=(0.25, 0.5, 1.0))
    specs = W.make_specs(rows)
    print(f"plain logs: {len(specs)} sims", flush=True)
    compare(gpu.run_log(logs, specs), oracle_lib.run_log(logs, specs), specs, "plain logs")


def test_long_logs_compaction_and_ragged_tiles(gpu, oracle_lib):
    """Logs of a few thousand operators (storage scans over many 64-wide
    rounds with a ragged tail; thousands of evictions against a union-find
    pool of 2S + 64 nodes, so it is compacted repeatedly)."""
    logs = [W.random_log(5000 + s, n_steps=1500 + 700 * s, n_const=3, max_size=20, max_cost=7, max_in=3, keep=3)
            for s in range(3)]
    peaks = unlimited_peaks(oracle_lib, logs)
    rows = []
    for i, pk in enumerate(peaks):
        rows += rows_for(i, pk, i, [W.H_DTR, W.H_EQ, W.H_LRU, W.H_MSPS, W.h_family(W.C_EQCLASS, 1, 0)],
                         policies=(W.POLICY_EAGER, W.POLICY_IGNORE), fracs=(0.1, 0.15, 0.3))
    specs = W.make_specs(rows)
    s_max = max(len(brute_log.StorageProgram(L).size) for L in logs)
    print(f"long logs: {s_max} storages at most, {len(specs)} sims", flush=True)
    ref = oracle_lib.run_log(logs, specs)
    compare(gpu.run_log(logs, specs), ref, specs, "long logs")
    compare(gpu.run_log(logs, specs, flags=gpu.OPT_LOG_NO_LDS), ref, specs, "long logs, device memory")
    # union-find nodes are created per eviction from a pool of 2 S_max + 64
    eq = [k for k in range(len(specs)) if specs["heuristic"][k] in UF]
    assert max(int(ref["n_evictions"][k] + ref["n_eager_evictions"][k]) for k in eq) > 3 * (2 * s_max + 64)


def test_empty_and_degenerate_logs(gpu, oracle_lib):
    b = W.LogBuilder("consts")
    c = [b.fresh() for _ in range(3)]
    for k, t in enumerate(c):
        b.constant(t, 3 + k)
    b.release(c[1])
    consts = b.build()
    empty = W.LogBuilder("empty").build()
    b = W.LogBuilder("one")
    x = b.fresh()
    b.call([], [x], 4, [5], [-1])
    one = b.build()
    logs = [empty, consts, one, W.random_log(9, n_steps=3, n_const=0)]
    rows = []
    for i in range(len(logs)):
        for h in HS:
            for policy in (W.POLICY_EAGER, W.POLICY_IGNORE, W.POLICY_BANISH):
                if policy == W.POLICY_BANISH and h in UF:
                    continue
                for bud in (0, 1, 4, 7, 12, W.BUDGET_UNLIMITED):
                    rows.append((i, h, bud, 5, policy))
    specs = W.make_specs(rows)
    compare(gpu.run_log(logs, specs), oracle_lib.run_log(logs, specs), specs, "degenerate logs")
    assert len(gpu.run_log(logs, specs[:0])) == 0


def test_log_determinism_across_slot_counts(gpu):
    logs = [W.random_log(40 + s, n_steps=200) for s in range(6)]
    rows = [(i, h, 20 + 7 * i, 3, W.POLICY_EAGER) for i in range(6) for h in HS]
    specs = W.make_specs(rows)
    a = gpu.run_log(logs, specs, slots=3)
    b = gpu.run_log(logs, specs, slots=500)
    c = gpu.run_log(logs, specs)
    assert a.tobytes() == b.tobytes() == c.tobytes()


def test_resnet_log_config_sampled(gpu, oracle_lib):
    """The PyTorch-style ResNet log (every instruction kind but COPYFROM, at
    its benchmark size): every 8th replay of the 1536 against the oracle."""
    wl = W.make_config("resnet50log")
    specs = wl.specs[::8]
    print(f"resnet log: {len(specs)} sims", flush=True)
    compare(gpu.run_log(wl.traces, specs), oracle_lib.run_log(wl.traces, specs), specs, "resnet50log")


def test_resnet_log_full_batch_properties(gpu):
    """All 1536 replays of the ResNet log in one launch, against properties
    that hold at any size: a finished replay runs every operator (CALL,
    MUTATE, CONSTANT) once at its listed cost, plus its rematerializations,
    within its budget."""
    wl = W.make_config("resnet50log")
    L = wl.traces[0]
    kind, value = np.asarray(L.kind), np.asarray(L.value)
    n_ops = int(np.isin(kind, [W.LOG_CALL, W.LOG_MUTATE, W.LOG_CONSTANT]).sum())
    base = int(value[np.isin(kind, [W.LOG_CALL, W.LOG_MUTATE])].sum())
    got = gpu.run_log(wl.traces, wl.specs)
    ok = got["status"] == 0
    assert ok.any() and (~ok).any()
    assert (got["total_cost"] == got["base_cost"] + got["remat_cost"]).all()
    assert (got["base_cost"][ok] == base).all()
    assert (got["n_executed_ops"][ok] == n_ops + got["n_remats"][ok]).all()
    assert (got["peak_memory"][ok] <= wl.specs["budget"][ok]).all()
    assert (got["failed_op"][ok] == -1).all() and (got["failed_op"][~ok] >= 0).all()


def test_workgroup_shapes_of_the_lds_variant(gpu, oracle_lib):
    """Logs of growing size take 4, 2 and 1 waves per workgroup (helper waves
    in the walk scans while the LDS holds their bitsets and stacks), then the
    device-memory variant; each shape against the oracle."""
    seen = set()
    for n_steps in (1500, 2300, 2500, 2700, 2900, 3100, 3600):
        L = W.random_log(6000 + n_steps, n_steps=n_steps, n_const=3, max_size=20, max_cost=7, max_in=3, keep=3)
        pk = unlimited_peaks(oracle_lib, [L])[0]
        rows = [(0, h, max(1, int(pk * f)), 11, W.POLICY_EAGER) for h in (W.H_DTR, W.H_MSPS, W.H_EQ)
                for f in (0.15, 0.4)]
        specs = W.make_specs(rows)
        sim = gpu.Simulator(None, specs, logs=[L])
        info = sim.launch_info()
        sim.run()
        got = sim.results()
        sim.close()
        shape = (info["waves_per_group"], info["lds_bytes"] > 0)
        print(f"log of {n_steps} steps: {info}", flush=True)
        seen.add(shape)
        compare(got, oracle_lib.run_log([L], specs), specs, f"log of {n_steps} steps, {info}")
    assert {(4, True), (2, True), (1, True), (1, False)} <= seen, seen


def test_more_storages_than_16_bit_ids(gpu, oracle_lib):
    """A log of 66000 storages (the Appendix A chain of 33000 layers written as
    a log): its neighbour ids do not fit the LDS variant's 16 bits, so it
    replays from device memory."""
    L = W.log_from_trace(W.chain_trace(33000))
    pk = W.log_peak(L)
    rows = [(0, h, int(pk * f), 3, W.POLICY_EAGER) for h in (W.H_LRU, W.H_EQ, W.H_SIZE) for f in (0.97, 0.99)]
    rows += [(0, h, int(pk * 0.99), 3, W.POLICY_EAGER) for h in (W.H_DTR, W.H_MSPS)]
    specs = W.make_specs(rows)
    sim = gpu.Simulator(None, specs, logs=[L])
    info = sim.launch_info()
    sim.run()
    got = sim.results()
    sim.close()
    print(f"66000-storage log: {info}", flush=True)
    assert info["lds_bytes"] == 0 and info["waves_per_group"] == 1
    compare(got, oracle_lib.run_log([L], specs), specs, "66000-storage chain log")


def test_wide_operators_as_logs(gpu, oracle_lib):
    """Operators with up to ~180 inputs and storages read by up to ~240
    operators, written as logs (inputs checked over several 64-lane chunks)."""
    logs, rows = [], []
    for s in range(3):
        tr = W.random_program(900 + s, n_ops=260, n_const=4, max_in=130, backward=s % 2 == 0, max_size=9,
                              max_cost=6)
        logs.append(W.log_from_trace(tr))
        rows += rows_for(s, W.natural_peak(tr), s, HS, policies=(W.POLICY_EAGER, W.POLICY_BANISH),
                         fracs=(0.8, 0.95, 0.995))
    specs = W.make_specs(rows)
    print(f"wide logs: {len(specs)} sims", flush=True)
    compare(gpu.run_log(logs, specs), oracle_lib.run_log(logs, specs), specs, "wide logs")


def test_deep_rematerialization_chain_logs(gpu, oracle_lib):
    """The Appendix A chain written as logs, at 700 layers (walk state in LDS)
    and 2000 layers (device memory): operator-call stacks about N frames deep
    at budget 4."""
    import math
    for N in (700, 2000):
        L = W.log_from_trace(W.chain_trace(N))
        rows = [(0, h, 2 * math.ceil(math.sqrt(N)), 3) for h in (W.H_DTR, W.H_EQ, W.H_ESTAR, W.H_MSPS)]
        rows += [(0, h, 4, 3) for h in (W.H_EQ, W.H_LRU)]
        specs = W.make_specs(rows)
        sim = gpu.Simulator(None, specs, logs=[L])
        info = sim.launch_info()
        sim.run()
        got = sim.results()
        sim.close()
        print(f"chain log of {N} layers: {info}", flush=True)
        compare(got, oracle_lib.run_log([L], specs, threads=16), specs, f"chain log {N}")


def test_resnet_log_policies(gpu, oracle_lib):
    """Ignoring releases and banishing on the PyTorch-style ResNet log (views,
    in-place operators, constants), at 8 budgets spread over its benchmark
    range, for the heuristics that take banishing."""
    wl = W.make_config("resnet50log")
    b = sorted(set(int(x) for x in wl.specs["budget"]))
    rows = [(0, h, b[len(b) * q // 8], 17 + h, pol) for q in range(8)
            for h in (W.H_DTR, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_MSPS)
            for pol in (W.POLICY_IGNORE, W.POLICY_BANISH)]
    specs = W.make_specs(rows)
    print(f"resnet log policies: {len(specs)} sims", flush=True)
    compare(gpu.run_log(wl.traces, specs), oracle_lib.run_log(wl.traces, specs, threads=16), specs,
            "resnet log policies")


def test_resnet_log_search_approximations(gpu, oracle_lib):
    """The search approximations on the ResNet log (a pool of up to ~1300
    storages; the LDS variant's walk scans with sampled candidate lists) at 5
    budgets, under h_DTR, h_DTR^eq and h_LRU."""
    wl = W.make_config("resnet50log")
    b = sorted(set(int(x) for x in wl.specs["budget"]))
    flags = (W.SEARCH_IGNORE_SMALL, W.SEARCH_SAMPLE, W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE)
    rows = [(0, h, b[len(b) * q // 6], 23 + h, W.POLICY_EAGER, sf) for q in range(1, 6)
            for h in (W.H_DTR, W.H_EQ, W.H_LRU) for sf in flags]
    specs = W.make_specs(rows)
    print(f"resnet log search: {len(specs)} sims", flush=True)
    compare(gpu.run_log(wl.traces, specs), oracle_lib.run_log(wl.traces, specs, threads=16), specs,
            "resnet log search")
