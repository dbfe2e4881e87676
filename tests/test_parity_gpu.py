"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle,
field by field and bit-exact (every quantity is an integer)."""
import math
import os

import numpy as np
import pytest

from paper_2006_09616_amd import workloads as W

pytestmark = pytest.mark.gpu

FIELDS = ["total_cost", "base_cost", "remat_cost", "peak_memory", "final_memory", "n_executed_ops",
          "n_remats", "n_evictions", "n_eager_evictions", "n_scores", "n_nbr_visits", "n_adj_visits",
          "status", "failed_op"]


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2006_09616_amd import dtr as D
    D.lib()
    return D


def compare(gpu_res, ref, specs, label):
    bad = []
    for k in range(len(specs)):
        for f in FIELDS:
            if int(gpu_res[f][k]) != int(ref[f][k]):
                bad.append((k, f, int(gpu_res[f][k]), int(ref[f][k]), tuple(specs[k])))
                break
    assert not bad, f"{label}: {len(bad)}/{len(specs)} differ; first: {bad[:4]}"


def specs_of(rows):
    return W.make_specs(rows)


def test_chain_all_heuristics(gpu, oracle_lib):
    traces = [W.chain_trace(N) for N in (2, 3, 8, 32, 100)]
    rows = []
    for i, tr in enumerate(traces):
        N = tr.n_ops // 2
        for h in range(7):
            for B in sorted({1, 2, 3, 4, max(3, N // 4), N, 2 * N, W.BUDGET_UNLIMITED}):
                rows.append((i, h, B, 77 + len(rows)))
    specs = specs_of(rows)
    print(f"chain batch: {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "chains")


@pytest.mark.parametrize("seed0", [0, 1000])
def test_random_programs(gpu, oracle_lib, seed0):
    traces = []
    rows = []
    for s in range(seed0, seed0 + 60):
        tr = W.random_program(s, n_ops=5 + (s * 7) % 120, n_const=s % 5, backward=s % 2 == 0,
                              max_in=1 + s % 5, max_size=1 + s % 30, max_cost=1 + s % 9,
                              window=None if s % 3 else 16)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for h in range(7):
            for frac in (0.2, 0.35, 0.5, 0.75, 1.0):
                rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s * 131 + h))
    specs = specs_of(rows)
    print(f"random batch: {len(traces)} traces, {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "random")


def test_msps_and_ablation_family(gpu, oracle_lib):
    """h_MSPS and every member of h'(s, m, c) on random programs."""
    traces = []
    rows = []
    hs = [W.H_MSPS] + W.ALL_FAMILY
    for s in range(40):
        tr = W.random_program(500 + s, n_ops=10 + (s * 13) % 90, n_const=s % 4, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + s % 20, max_cost=1 + s % 7)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for h in hs:
            for frac in (0.25, 0.5, 0.8):
                rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s * 37 + h))
    specs = specs_of(rows)
    print(f"family batch: {len(traces)} traces, {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "family")


def test_deallocation_policies(gpu, oracle_lib):
    """Ignoring releases and banishing, every heuristic the policy allows."""
    uf = {W.H_EQ} | {W.h_family(W.C_EQCLASS, s, m) for s in (0, 1) for m in (0, 1)}
    traces = []
    rows = []
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS,
          W.h_family(W.C_ESTAR, 1, 0), W.h_family(W.C_NONE, 0, 0)]
    for s in range(40):
        tr = W.random_program(900 + s, n_ops=10 + (s * 11) % 100, n_const=1 + s % 4, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + s % 20, max_cost=1 + s % 7)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for policy in (W.POLICY_IGNORE, W.POLICY_BANISH):
            for h in hs:
                if policy == W.POLICY_BANISH and h in uf:
                    continue
                for frac in (0.3, 0.6, 1.0):
                    rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s * 31 + h, policy))
    n_chain = len(traces)
    traces.append(W.chain_trace(200))
    for B in (2 * 15, 40, 80):
        rows.append((n_chain, W.H_ESTAR, B, 0, W.POLICY_BANISH))
        rows.append((n_chain, W.H_DTR, B, 0, W.POLICY_BANISH))
    specs = specs_of(rows)
    print(f"policy batch: {len(traces)} traces, {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "policies")


def test_search_approximations(gpu, oracle_lib):
    """Ignoring small candidates and sampling the pool, with every heuristic
    class, on random programs and on the ResNet trace."""
    traces = []
    rows = []
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_RAND, W.H_MSPS]
    flags = (W.SEARCH_IGNORE_SMALL, W.SEARCH_SAMPLE, W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE)
    for s in range(30):
        tr = W.random_program(1300 + s, n_ops=20 + (s * 17) % 120, n_const=s % 4, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + (s * 13) % 200, max_cost=1 + s % 7)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for search in flags:
            for h in hs:
                for frac in (0.3, 0.6):
                    rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s * 53 + h, W.POLICY_EAGER, search))
    rn = W.make_config("resnet50blk")
    traces.append(rn.traces[0])
    for search in flags:
        for h in (W.H_DTR, W.H_EQ, W.H_LRU):
            for k in range(0, 256, 32):
                rows.append((len(traces) - 1, h, int(rn.specs["budget"][k]), 7 + k, W.POLICY_EAGER, search))
    specs = specs_of(rows)
    print(f"search batch: {len(traces)} traces, {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "search")


def test_empty_and_degenerate(gpu, oracle_lib):
    empty = W.Trace("empty", np.zeros(0, np.int64), np.zeros(0, np.uint8), np.zeros(0, np.int32),
                    np.zeros(0, np.int64), np.zeros(1, np.int64), np.zeros(0, np.int32))
    consts = W.Trace("consts", np.array([5, 7], np.int64), np.array([1, 3], np.uint8),
                     np.zeros(0, np.int32), np.zeros(0, np.int64), np.zeros(1, np.int64),
                     np.zeros(0, np.int32))
    single = W.Trace("single", np.array([4], np.int64), np.array([2], np.uint8), np.array([0], np.int32),
                     np.array([3], np.int64), np.array([0, 0], np.int64), np.zeros(0, np.int32))
    traces = [empty, consts, single, W.chain_trace(1)]
    rows = []
    for i in range(len(traces)):
        for h in range(7):
            for b in (0, 1, 4, 11, 12, W.BUDGET_UNLIMITED):
                rows.append((i, h, b, 5))
    specs = specs_of(rows)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs), specs, "degenerate")
    assert len(gpu.run(traces, specs[:0])) == 0


def test_chain32_config(gpu, oracle_lib):
    w = W.make_config("chain32")
    compare(gpu.run(w.traces, w.specs), oracle_lib.run(w.traces, w.specs), w.specs, "chain32")


def test_resnet_config(gpu, oracle_lib):
    w = W.make_config("resnet50blk")
    print(f"resnet: {w.n_sims} sims", flush=True)
    compare(gpu.run(w.traces, w.specs), oracle_lib.run(w.traces, w.specs), w.specs, "resnet")


def test_transformer_config(gpu, oracle_lib):
    w = W.make_config("transformer12")
    print(f"transformer: {w.n_sims} sims", flush=True)
    compare(gpu.run(w.traces, w.specs), oracle_lib.run(w.traces, w.specs), w.specs, "transformer")


def test_treelstm_subset(gpu, oracle_lib):
    w = W.make_config("treelstm4096", n_trees=128)
    print(f"treelstm subset: {w.n_sims} sims", flush=True)
    compare(gpu.run(w.traces, w.specs), oracle_lib.run(w.traces, w.specs), w.specs, "treelstm128")


def test_determinism_across_slot_counts(gpu):
    """The mixed ResNet batch (three kernel groups): with 2 slots the groups
    run one after another over both, with 7 or more side by side on streams
    of their own over disjoint slots; the results are the same."""
    w = W.make_config("resnet50blk")
    a = gpu.run(w.traces, w.specs, slots=7)
    b = gpu.run(w.traces, w.specs, slots=1000)
    c = gpu.run(w.traces, w.specs)
    d = gpu.run(w.traces, w.specs, slots=2)
    assert a.tobytes() == b.tobytes() == c.tobytes() == d.tobytes()


def test_determinism_under_shuffled_order(gpu):
    """Each simulation's result depends on its spec alone: the batch shuffled
    (so simulations land in other slots, other workgroups and another dispatch
    order) gives the same result per simulation."""
    w = W.make_config("resnet50blk")
    t = W.make_config("treelstm4096", n_trees=64)
    for wl in (w, t):
        a = gpu.run(wl.traces, wl.specs)
        perm = np.random.default_rng(3).permutation(wl.n_sims)
        b = gpu.run(wl.traces, wl.specs[perm])
        assert a[perm].tobytes() == b.tobytes(), wl.name


def test_random_dag_replica_all_budgets(gpu, oracle_lib):
    """Random-DAG recipe (1-3 inputs from the previous 64 outputs, log-normal
    sizes) at 1000 forward ops, h_DTR at 12 budgets from 5% to 100%: the
    budget range of the full workload on a trace the oracle finishes."""
    w = W.config_random_dag(n_forward=1000, n_budgets=12)
    print(f"random dag replica: {w.n_sims} sims", flush=True)
    compare(gpu.run(w.traces, w.specs), oracle_lib.run(w.traces, w.specs), w.specs, "randdag1k")


def test_random_dag_full_size_goldens(gpu):
    """The full 100k-forward-op random DAG (200k ops, h_DTR with exact e*)
    against stored oracle results (tests/golden/randdag100k_oracle.json,
    written by a script that calls only the oracle): the stored budgets from
    19% to 100% of the peak, in one launch of the batch's kernel shape (8
    wavefronts per workgroup; about 130 s).  The two lowest (5% and 10%) run
    for minutes: test_random_dag_lowest_budget_goldens, on request."""
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "randdag100k_oracle.json")))
    w = W.make_config("randdag100k")
    assert w.traces[0].digest() == g["trace_sha256"]
    rows = [r for r in g["sims"] if r["index"] >= 154]
    pick = np.array([r["index"] for r in rows])
    specs = w.specs[pick]
    print(f"random dag full size: budget indices {pick.tolist()}", flush=True)
    got = gpu.run(w.traces, specs)
    bad = [(r["index"], f, int(got[f][k]), v) for k, r in enumerate(rows) for f, v in r["result"].items()
           if int(got[f][k]) != v]
    assert not bad, f"randdag100k goldens: {bad[:6]}"


@pytest.mark.skipif(os.environ.get("DTR_LONG_TESTS") != "1",
                    reason="runs about 8 minutes on one MI355X; set DTR_LONG_TESTS=1 (run with -s to see its progress)")
def test_random_dag_lowest_budget_goldens(gpu):
    """The full random DAG at its two lowest stored budgets (5% and 10% of the
    peak), against the stored oracle results, in one launch that runs for
    minutes; progress lines come from the launch's own operation counter."""
    import json
    import time
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "randdag100k_oracle.json")))
    w = W.make_config("randdag100k")
    assert w.traces[0].digest() == g["trace_sha256"]
    rows = [r for r in g["sims"] if r["index"] < 154]
    pick = np.array([r["index"] for r in rows])
    print(f"random dag full size: budget indices {pick.tolist()}", flush=True)
    sim = gpu.Simulator(w.traces, w.specs[pick])
    t0 = time.time()
    sim.run()
    while not sim.done():
        time.sleep(20)
        print(f"  {time.time() - t0:5.0f} s: {sim.progress()} operations executed", flush=True)
    got = sim.results()
    sim.close()
    bad = [(r["index"], f, int(got[f][k]), v) for k, r in enumerate(rows) for f, v in r["result"].items()
           if int(got[f][k]) != v]
    assert not bad, f"randdag100k goldens: {bad[:6]}"


def test_progress_counter(gpu):
    """dtr_sim_progress after a run: each walk-heuristic simulation counted in
    whole steps of 4096 executed operations, the others not at all."""
    rd = W.config_random_dag(n_forward=3000, n_budgets=6)
    rn = W.make_config("resnet50blk")
    traces = [rd.traces[0], rn.traces[0]]
    rows = [(0, W.H_DTR, int(b), 0) for b in rd.specs["budget"][2:]]
    rows += [(0, h, int(rd.specs["budget"][3]), 0) for h in (W.H_EQ, W.H_LRU, W.H_ESTAR, W.H_MSPS)]
    rows += [(1, h, int(rn.specs["budget"][k]), 0) for k in (0, 100) for h in (W.H_DTR, W.H_EQ)]
    specs = specs_of(rows)
    sim = gpu.Simulator(traces, specs)
    assert sim.progress() == 0
    sim.run()
    res = sim.results()
    walk = np.isin(specs["heuristic"], [W.H_DTR, W.H_ESTAR, W.H_MSPS])
    expect = int((res["n_executed_ops"][walk] // 4096 * 4096).sum())
    assert expect > 0
    assert sim.progress() == expect
    sim.run_static()                    # the counter of the static working memory
    assert sim.results().tobytes() == res.tobytes()
    assert sim.progress() == expect
    sim.close()


def test_treelstm_full_batch_sampled(gpu, oracle_lib):
    """The full TreeLSTM batch (4096 traces x 8 budgets, 32768 simulations) in
    one launch, as the benchmark times it: every simulation checked against
    properties that hold at any size, every 257th against the oracle (a stride
    coprime to the 8 budgets per tree, so every budget level is sampled)."""
    w = W.make_config("treelstm4096")
    print(f"treelstm full batch: {w.n_sims} sims", flush=True)
    got = gpu.run(w.traces, w.specs)
    ok = got["status"] == 0
    assert (got["total_cost"] == got["base_cost"] + got["remat_cost"]).all()
    assert (got["peak_memory"][ok] <= w.specs["budget"][ok]).all()
    assert (got["final_memory"][ok] <= w.specs["budget"][ok]).all()
    # a finished simulation executes every trace operation once, plus its rematerializations
    base = np.array([int(t.op_cost.sum()) for t in w.traces])[w.specs["trace"]]
    n_ops = np.array([t.n_ops for t in w.traces])[w.specs["trace"]]
    assert (got["base_cost"][ok] == base[ok]).all()
    assert (got["n_executed_ops"][ok] == n_ops[ok] + got["n_remats"][ok]).all()
    assert (got["failed_op"][ok] == -1).all() and (got["failed_op"][~ok] >= 0).all()
    assert set(np.unique(got["status"]).tolist()) <= {0, 1}
    pick = np.arange(0, w.n_sims, 257)
    assert len(set((pick % 8).tolist())) == 8
    sub = w.specs[pick]
    compare(got[pick], oracle_lib.run(w.traces, sub, threads=16), sub, "treelstm4096-sampled")


def _wide_programs():
    """Programs whose operators read up to ~180 inputs and whose tensors feed
    up to ~240 operators: input locking, rematerialization checks, unlocking,
    neighbour caches, merges and walks all run over several 64-lane chunks."""
    return [W.random_program(900 + s, n_ops=260, n_const=4, max_in=130, backward=s % 2 == 0, max_size=9,
                             max_cost=6) for s in range(3)]


def _wide_rows(traces):
    rows = []
    for i, tr in enumerate(traces):
        pk = W.natural_peak(tr)
        for h in range(8):
            for pol in (W.POLICY_EAGER, W.POLICY_BANISH):
                if pol == W.POLICY_BANISH and h == W.H_EQ:
                    continue
                for f in (0.8, 0.95, 0.995):
                    rows.append((i, h, int(pk * f), 7 + i, pol))
    return rows


def test_wide_operators(gpu, oracle_lib):
    trs = _wide_programs()
    specs = specs_of(_wide_rows(trs))
    print(f"wide operators: {len(specs)} sims", flush=True)
    compare(gpu.run(trs, specs), oracle_lib.run(trs, specs), specs, "wide operators")


def test_deep_rematerialization_chain(gpu, oracle_lib):
    """The Appendix A chain at 2000 layers: at budget 2*ceil(sqrt(N)) under
    the neighbourhood heuristics, and at budget 4 under h_DTR^eq, h_LRU and
    h_size, where backward steps rematerialize the forward chain from its start
    (remat stacks about N frames deep, ~1M rematerializations)."""
    N = 2000
    tr = W.chain_trace(N)
    rows = [(0, h, 2 * math.ceil(math.sqrt(N)), 3) for h in (W.H_DTR, W.H_EQ, W.H_LRU, W.H_ESTAR, W.H_MSPS)]
    rows += [(0, h, 4, 3) for h in (W.H_EQ, W.H_LRU, W.H_SIZE)]
    specs = specs_of(rows)
    print(f"deep chain: {len(specs)} sims", flush=True)
    ref = oracle_lib.run([tr], specs, threads=16)
    compare(gpu.run([tr], specs), ref, specs, "deep chain")
    assert int(ref["n_remats"].max()) > 500_000


def test_search_approximations_on_large_pools(gpu, oracle_lib):
    """The search approximations on TreeLSTM traces whose pools hold hundreds
    to thousands of candidates (scan rounds beyond the LDS head), under
    h_DTR^eq and h_LRU, at the 43%, 54% and 89% budgets of each tree."""
    w = W.make_config("treelstm4096", n_trees=12)
    flags = (W.SEARCH_IGNORE_SMALL, W.SEARCH_SAMPLE, W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE)
    rows = [(int(w.specs["trace"][k]), h, int(w.specs["budget"][k]), 11 + k, W.POLICY_EAGER, sf)
            for k in range(len(w.specs)) if k % 8 in (2, 3, 6) for sf in flags for h in (W.H_EQ, W.H_LRU)]
    specs = specs_of(rows)
    print(f"search on large pools: {len(specs)} sims", flush=True)
    ref = oracle_lib.run(w.traces, specs, threads=16)
    compare(gpu.run(w.traces, specs), ref, specs, "search, large pools")
    assert float(ref["n_scores"].sum()) / max(1, int(ref["n_evictions"].sum())) > 256


def test_policies_on_model_traces(gpu, oracle_lib):
    """Ignoring releases and banishing on the ResNet and transformer traces
    (pools of hundreds of tensors, long release lists), every heuristic that
    takes banishing, at 8 budgets spread over each trace's benchmark range."""
    traces, rows = [], []
    for name in ("resnet50blk", "transformer12"):
        w = W.make_config(name)
        traces.append(w.traces[0])
        b = sorted(set(int(x) for x in w.specs["budget"]))
        for bb in (b[len(b) * q // 8] for q in range(8)):
            for h in (W.H_DTR, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS):
                for pol in (W.POLICY_IGNORE, W.POLICY_BANISH):
                    rows.append((len(traces) - 1, h, bb, 17 + h, pol))
    specs = specs_of(rows)
    print(f"policies on model traces: {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs), oracle_lib.run(traces, specs, threads=16), specs, "policies, model traces")


def test_clock_overflow_goldens(gpu, oracle_lib):
    """The clock guard reached in a trace operation, in a rematerialization
    inside one, and in the output condition (hand-derived goldens), under
    every heuristic class and family member, bit-exact against the oracle."""
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "clock_overflow.json")))
    traces = [W.plain_chain(c["chain"]["n_ops"], g["cost"], c["chain"]["last_reads_first"], c["chain"]["required"])
              for c in g["cases"]]
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS] + W.ALL_FAMILY
    rows = [(i, h, c["budget"], 9 + h) for i, c in enumerate(g["cases"]) for h in hs]
    specs = specs_of(rows)
    got = gpu.run(traces, specs)
    compare(got, oracle_lib.run(traces, specs), specs, "clock overflow")
    for k, (i, h, _, _) in enumerate(rows):
        for f, v in g["cases"][i]["expected"].items():
            assert int(got[f][k]) == v, (g["cases"][i]["name"], h, f)


def test_shared_weight_chains(gpu, oracle_lib):
    """A chain whose every operator also reads one weight: at budgets 5-8 the
    rematerialization stack holds the weight hundreds of times over (up to ~590
    nested frames at N=600), as a constant and as an evictable operator output
    (twice the size of a layer), bit-exact against the oracle."""
    traces = [W.shared_weight_chain(600), W.shared_weight_chain(600, weight_size=2, constant=False),
              W.shared_weight_chain(1000)]
    rows = []
    for i in range(len(traces)):
        for h in (W.H_LRU, W.H_EQ, W.H_DTR, W.H_SIZE, W.H_LOCAL, W.H_MSPS):
            for b in (5, 6, 7, 8) if i < 2 else (6,):
                rows.append((i, h, b + (i == 1), 21 + i))
    specs = specs_of(rows)
    print(f"shared weight chains: {len(specs)} sims", flush=True)
    ref = oracle_lib.run(traces, specs, threads=8)
    assert (ref["status"] == 0).all()
    compare(gpu.run(traces, specs), ref, specs, "shared weight chains")


def test_near_ties_at_large_magnitude(gpu, oracle_lib):
    """Scores that tie exactly or differ by less than 2^-16 (down to about
    2^-39) at sizes near 2^35, costs up to 2^28 and staleness near 2^39:
    decisions the kernel's float estimate cannot separate, which it must
    hand to the exact 128-bit comparison (ties to the smaller id)."""
    traces = [W.near_tie_program(s) for s in range(16)]
    hs = [W.H_LOCAL, W.H_SIZE, W.H_LRU, W.H_EQ, W.H_DTR, W.H_ESTAR, W.H_MSPS,
          W.h_family(W.C_LOCAL, 1, 0), W.h_family(W.C_EQCLASS, 0, 1), W.h_family(W.C_NONE, 1, 1)]
    rows = [(i, h, b, i) for i, t in enumerate(traces) for h in hs for b in W.near_tie_budgets(t)]
    specs = specs_of(rows)
    print(f"near ties: {len(specs)} sims", flush=True)
    ref = oracle_lib.run(traces, specs)
    assert (ref["status"] == 0).all() and int(ref["n_evictions"].min()) > 0
    compare(gpu.run(traces, specs), ref, specs, "near ties")


WALK_H = [W.H_DTR, W.H_ESTAR, W.H_MSPS, W.h_family(W.C_ESTAR, 1, 0), W.h_family(W.C_ESTAR, 0, 0)]


@pytest.mark.parametrize("waves,small", [(1, True), (2, False), (8, False), (8, True)])
def test_walk_workgroup_shapes(gpu, oracle_lib, waves, small):
    """The e* / e_R walks with 1, 2 or 8 wavefronts sharing each eviction
    scan, and with lane queues of 16 members (so that larger neighbourhoods
    take the whole-wavefront walk), on random programs, the ResNet trace and
    a chain of 300 layers, every walk heuristic and policy."""
    traces, rows = [], []
    for s in range(24):
        tr = W.random_program(2100 + s, n_ops=20 + (s * 23) % 150, n_const=s % 3, backward=s % 2 == 0,
                              max_in=1 + s % 4, max_size=1 + s % 25, max_cost=1 + s % 9)
        traces.append(tr)
        peak = W.natural_peak(tr)
        for h in WALK_H:
            for frac in (0.25, 0.5, 0.8):
                rows.append((len(traces) - 1, h, max(1, int(peak * frac)), s, W.POLICY_EAGER if s % 3 else W.POLICY_BANISH))
    rn = W.make_config("resnet50blk")
    traces.append(rn.traces[0])
    for k in range(0, 256, 51):
        rows.append((len(traces) - 1, W.H_DTR, int(rn.specs["budget"][k]), 0))
    traces.append(W.chain_trace(300))
    for b in (2 * 18, 60):
        for h in (W.H_DTR, W.H_ESTAR, W.H_MSPS):
            rows.append((len(traces) - 1, h, b, 0))
    specs = specs_of(rows)
    flags = gpu.opt_walk_waves(waves) | (gpu.OPT_WALK_QUEUE_SMALL if small else 0)
    print(f"walk shapes {waves} waves, small queues {small}: {len(specs)} sims", flush=True)
    ref = oracle_lib.run(traces, specs)
    if small:
        assert int(ref["n_nbr_visits"].max()) > 0
    compare(gpu.run(traces, specs, flags=flags), ref, specs, f"walk {waves} waves small={small}")


_EQ_BATCH = {}


def _eq_batch(oracle_lib):
    """TreeLSTM traces at tight budgets (pools of several rounds), the ResNet
    trace, wide operators (overflowed neighbour caches) and random programs,
    under h_DTR^eq and the union-find members of the h' family; the oracle's
    results computed once."""
    if not _EQ_BATCH:
        tl = W.make_config("treelstm4096", n_trees=24)
        rn = W.make_config("resnet50blk")
        traces, rows = list(tl.traces), []
        for k in range(tl.n_sims):
            t, h, b, seed = (int(v) for v in tuple(tl.specs[k])[:4])
            rows.append((t, h, b, seed))
        traces.append(rn.traces[0])
        for k in range(0, 256, 37):
            rows.append((len(traces) - 1, W.H_EQ, int(rn.specs["budget"][k]), 0))
        for tr in _wide_programs()[:6]:
            traces.append(tr)
            peak = W.natural_peak(tr)
            for frac in (0.3, 0.6):
                rows.append((len(traces) - 1, W.H_EQ, max(1, int(peak * frac)), 0))
        for s in range(12):
            tr = W.random_program(3300 + s, n_ops=40 + (s * 37) % 200, n_const=s % 3, backward=True,
                                  max_in=1 + s % 5, max_size=1 + s % 30, max_cost=1 + s % 9)
            traces.append(tr)
            peak = W.natural_peak(tr)
            for h in (W.H_EQ, W.h_family(W.C_EQCLASS, 1, 0), W.h_family(W.C_EQCLASS, 0, 1),
                      W.h_family(W.C_EQCLASS, 0, 0)):
                rows.append((len(traces) - 1, h, max(1, int(peak * 0.35)), s))
        specs = specs_of(rows)
        _EQ_BATCH.update(traces=traces, specs=specs, ref=oracle_lib.run(traces, specs))
    return _EQ_BATCH["traces"], _EQ_BATCH["specs"], _EQ_BATCH["ref"]


@pytest.mark.parametrize("slots", [1, 5, 0])
def test_eq_wavefront_slots(gpu, oracle_lib, slots):
    """The exact h_DTR^eq kernel runs a simulation per wavefront, four
    wavefronts (slots) to a workgroup: one slot, five (a workgroup with one
    slot used and three idle wavefronts) and the default count."""
    traces, specs, ref = _eq_batch(oracle_lib)
    print(f"h_DTR^eq batch, slots={slots}: {len(specs)} sims", flush=True)
    compare(gpu.run(traces, specs, slots=slots), ref, specs, f"eq slots={slots}")
