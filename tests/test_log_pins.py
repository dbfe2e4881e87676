"""Pins of the log-replay oracle (operator logs, Appendix C.6): reduction to
the trace simulator on plain programs, hand-worked logs whose results follow
from the definitions (views, multi-output rematerialization, mutation,
reference counting), and a second, independently written Python machine."""
import numpy as np
import pytest

import brute_log
from paper_2006_09616_amd import workloads as W

FIELDS = ["total_cost", "base_cost", "remat_cost", "peak_memory", "final_memory", "n_executed_ops", "n_remats",
          "n_evictions", "n_eager_evictions", "n_scores", "status", "failed_op"]


def run_log(O, L, h, b, seed=0, policy=W.POLICY_EAGER, search=0):
    return O.run_log([L], W.make_specs([(0, h, b, seed, policy, search)]))[0]


def test_plain_programs_reduce_to_the_trace_simulator(oracle_lib):
    """A program written as a log (one storage per tensor, single outputs, no
    views) replays exactly like the trace."""
    O = oracle_lib
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_SIZE, W.H_RAND, W.H_ESTAR, W.H_MSPS,
          W.h_family(W.C_EQCLASS, 0, 1)]
    for seed in range(30):
        tr = W.random_program(seed, n_ops=12 + seed % 25, n_const=0, backward=seed % 2 == 0, permute_ids=False,
                              max_size=9, max_cost=6)
        L = W.log_from_trace(tr)
        peak = W.natural_peak(tr)
        rows = []
        for h in hs:
            for policy in (W.POLICY_EAGER, W.POLICY_IGNORE, W.POLICY_BANISH):
                if policy == W.POLICY_BANISH and h in (W.H_EQ, W.h_family(W.C_EQCLASS, 0, 1)):
                    continue
                for search in (0, W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE):
                    for b in (peak // 3, peak // 2, peak):
                        rows.append((0, h, b, seed, policy, search))
        specs = W.make_specs(rows)
        a, c = O.run([tr], specs), O.run_log([L], specs)
        for f in FIELDS:
            assert np.array_equal(a[f], c[f]), (seed, f)


def test_constants_become_nullary_operators(oracle_lib):
    """Constants in a log are cost-0 nullary operators of pinned storages: the
    replay matches the trace except for those extra operations."""
    O = oracle_lib
    for seed in range(20):
        tr = W.random_program(seed, n_ops=20 + seed, n_const=1 + seed % 4, backward=False, permute_ids=False,
                              max_size=9)
        n_const = int(((tr.tensor_flags & W.FLAG_CONSTANT) != 0).sum())
        const_mem = int(tr.tensor_size[(tr.tensor_flags & W.FLAG_CONSTANT) != 0].sum())
        L = W.log_from_trace(tr)
        peak = W.natural_peak(tr)
        for h in (W.H_DTR, W.H_LRU):
            for b in sorted({max(const_mem, peak // 2), peak}):
                a = O.run([tr], W.make_specs([(0, h, b, seed)]))[0]
                c = run_log(O, L, h, b, seed)
                if a["status"] != 0:
                    continue
                for f in FIELDS:
                    want = int(a[f]) + (n_const if f == "n_executed_ops" else 0)
                    assert int(c[f]) == want, (seed, h, b, f)


def _log(build):
    b = W.LogBuilder("pin")
    b.next_name = 100
    build(b)
    return b.build()


def test_views_share_their_storage(oracle_lib):
    """A view costs no memory and keeps its storage referenced."""
    def build(b):
        b.call([], [0], 1, [10], [-1])
        b.call([0], [1], 1, [99], [0])         # a view of 0: its MEMORY size is ignored
        b.release(0)
    r = run_log(oracle_lib, _log(build), W.H_DTR, W.BUDGET_UNLIMITED)
    assert (r["status"], r["peak_memory"], r["final_memory"], r["n_eager_evictions"]) == (0, 10, 10, 0)


def test_multi_output_remat_frees_the_duplicate(oracle_lib):
    """Worked by hand with h_size and budget 11: op0 makes a (2) and b (3);
    op2 evicts the larger, b; op3 reads a, b, d, so op0 runs again with a still
    resident: memory reaches 2+3 + 4 (d) + 2 (second copy of a) = 11, then the
    copy is freed."""
    def build(b):
        b.call([], [0, 1], 4, [2, 3], [-1, -1])    # a, b
        b.call([0], [2], 1, [4], [-1])             # c
        b.call([2], [3], 1, [4], [-1])             # d (evicts b)
        b.release(2)
        b.call([0, 1, 3], [4], 1, [1], [-1])       # e
    r = run_log(oracle_lib, _log(build), W.H_SIZE, 11)
    got = {f: int(r[f]) for f in FIELDS}
    assert got == dict(total_cost=11, base_cost=7, remat_cost=4, peak_memory=11, final_memory=10,
                       n_executed_ops=5, n_remats=1, n_evictions=1, n_eager_evictions=1,
                       n_scores=2, status=0, failed_op=-1)


def test_views_rerun_after_their_storage_returns(oracle_lib):
    """Budget 6: x (5) is evicted for y; after y's release, z reads the view v,
    so x's operator and then v's view operator run again."""
    def build(b):
        b.call([], [0], 3, [5], [-1])     # x
        b.call([0], [1], 1, [0], [0])     # v, a view of x
        b.release(0)
        b.call([], [2], 1, [5], [-1])     # y: evicts x
        b.release(2)
        b.call([1], [3], 1, [1], [-1])    # z reads v
    r = run_log(oracle_lib, _log(build), W.H_DTR, 6)
    got = {f: int(r[f]) for f in FIELDS}
    assert got == dict(total_cost=10, base_cost=6, remat_cost=4, peak_memory=6, final_memory=6,
                       n_executed_ops=6, n_remats=2, n_evictions=1, n_eager_evictions=1,
                       n_scores=1, status=0, failed_op=-1)


def test_mutation_clones_then_releases_the_original(oracle_lib):
    def build(b):
        b.call([], [0], 2, [4], [-1])
        b.mutate([0], [0], 1)
    r = run_log(oracle_lib, _log(build), W.H_DTR, W.BUDGET_UNLIMITED)
    assert (r["peak_memory"], r["final_memory"], r["n_executed_ops"], r["total_cost"],
            r["n_eager_evictions"]) == (8, 4, 2, 3, 1)


def test_copies_hold_references(oracle_lib):
    def build(b):
        b.call([], [0], 1, [3], [-1])
        b.copy(1, 0)
        b.release(0)                       # still referenced through the copy
        b.call([], [2], 1, [2], [-1])
        b.copyfrom(2, 1)                   # 2 now names x; its old tensor is dropped
    r = run_log(oracle_lib, _log(build), W.H_DTR, W.BUDGET_UNLIMITED)
    assert (r["peak_memory"], r["final_memory"], r["n_eager_evictions"]) == (5, 3, 1)


def test_matches_independent_python_machine(oracle_lib):
    O = oracle_lib
    hs = [W.H_DTR, W.H_EQ, W.H_LOCAL, W.H_LRU, W.H_RAND, W.H_ESTAR, W.H_MSPS, W.h_family(W.C_EQCLASS, 0, 1),
          W.h_family(W.C_NONE, 0, 0)]
    for seed in range(50):
        L = W.random_log(seed, 20 + seed % 40, n_const=seed % 4, max_size=6)
        total = sum(brute_log.StorageProgram(L).size)
        for h in hs:
            for policy in (W.POLICY_EAGER, W.POLICY_IGNORE, W.POLICY_BANISH):
                if policy == W.POLICY_BANISH and h in (W.H_EQ, W.h_family(W.C_EQCLASS, 0, 1)):
                    continue
                for b in (max(1, total // 5), max(1, total // 3), total):
                    r = run_log(O, L, h, b, seed, policy)
                    s = brute_log.simulate(L, b, h, seed, policy)
                    for k, v in s.items():
                        assert int(r[k]) == v, (seed, h, policy, b, k)


def test_malformed_logs_are_rejected(oracle_lib):
    O = oracle_lib
    bad = [
        lambda b: b.call([5], [0], 1, [1], [-1]),                          # unknown input name
        lambda b: (b.call([], [0], 1, [1], [-1]), b.call([], [0], 1, [1], [-1])),   # output name reused
        lambda b: (b.call([], [0], 1, [1], [-1]), b.release(0), b.release(0)),      # double release
        lambda b: (b.call([], [0], 1, [1], [-1]), b.call([], [1], 1, [1], [0])),    # view of a non-input
        lambda b: (b.call([], [0], 1, [1], [-1]), b.mutate([0], [3], 1)),           # mutates a non-input
        lambda b: (b.call([], [0], 1, [1], [-1]), b.call([0], [1, 1], 1, [1, 1], [0, 0])),  # output listed twice
    ]
    for build in bad:
        with pytest.raises(RuntimeError):
            run_log(O, _log(build), W.H_DTR, 10)


def test_storage_cost_sums_over_its_tensors(oracle_lib):
    """Appendix C.2 'Cost': cost(S) sums cost(op(t)) over every tensor t
    viewing S, so an operator returning a storage and a view of it counts
    twice.  A call returns a (4 units) and a view of a, at cost 3; a second
    call returns b (4 units) at cost 5; a third call needs 8 units under a
    budget of 12.  With c = c0 and staleness ablated (score c0/m), a's storage
    scores 6/4 and b's 5/4, so b is evicted (counting the call once would give
    3/4 and evict a).  c is released at once; the output condition then
    rematerializes b: total cost 3 + 5 + 1 + 5 = 14."""
    b = W.LogBuilder("shared-op")
    a, av, bb, c = b.fresh(), b.fresh(), b.fresh(), b.fresh()
    b.call([], [a, av], 3, [4, 4], [-1, a])
    b.call([], [bb], 5, [4], [-1])
    b.call([], [c], 1, [8], [-1])
    b.release(c)
    L = b.build()
    h = W.h_family(W.C_LOCAL, 0, 1)
    r = run_log(oracle_lib, L, h, 12)
    assert int(r["status"]) == 0
    assert (int(r["n_evictions"]), int(r["n_eager_evictions"]), int(r["n_remats"])) == (1, 1, 1)
    assert (int(r["remat_cost"]), int(r["total_cost"])) == (5, 14)
    assert int(r["peak_memory"]) == 12
    assert brute_log.simulate(L, 12, h, 0)["total_cost"] == 14


def test_storage_metadata_grows_with_its_views(oracle_lib):
    """Appendix C.2: the dependency graph and a storage's cost are those of the
    tensors that exist at the time (the cost changes when a view is made).
    a (4 units, cost 3) and b (4 units, cost 5) are made; a call of 8 units
    under a budget of 12 evicts one of them by c0/m (staleness ablated): a
    scores 3/4 and is evicted, because the view of a made afterwards (cost 10)
    does not exist yet (counting it would give a 13/4 and evict b).  The view
    then rematerializes a (cost 3): total 3 + 5 + 1 + 3 + 10 = 22."""
    b = W.LogBuilder("later-view")
    a, bb, c, av = b.fresh(), b.fresh(), b.fresh(), b.fresh()
    b.call([], [a], 3, [4], [-1])
    b.call([], [bb], 5, [4], [-1])
    b.call([], [c], 1, [8], [-1])
    b.release(c)
    b.call([a], [av], 10, [4], [a])
    L = b.build()
    h = W.h_family(W.C_LOCAL, 0, 1)
    r = run_log(oracle_lib, L, h, 12)
    assert int(r["status"]) == 0
    assert (int(r["n_evictions"]), int(r["n_remats"]), int(r["remat_cost"]), int(r["total_cost"])) == (1, 1, 3, 22)
    assert brute_log.simulate(L, 12, h, 0)["total_cost"] == 22
