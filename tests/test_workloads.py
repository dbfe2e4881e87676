"""Shape and validity checks of the seeded synthetic workloads."""
import math
import os

import numpy as np
import pytest

from paper_2006_09616_amd import workloads as W


def _valid(tr):
    defined = (tr.tensor_flags & W.FLAG_CONSTANT) != 0
    produced = np.zeros(tr.n_tensors, bool)
    for o in range(tr.n_ops):
        ins = tr.inputs(o)
        assert len(set(ins.tolist())) == len(ins)
        assert defined[ins].all()
        t = tr.op_output[o]
        assert not defined[t] and not produced[t]
        defined[t] = produced[t] = True
    assert defined.all()
    assert (tr.tensor_size >= 1).all() and (tr.op_cost >= 1).all()


def test_chain_matches_appendix_a_program():
    tr = W.chain_trace(32)
    _valid(tr)
    assert tr.n_ops == 64
    assert len(tr.op_inputs) == 93
    assert tr.inputs(32).tolist() == [30]          # grad of f_32 reads t_31
    assert tr.inputs(63).tolist() == [62]          # grad of f_1 reads grad of f_2
    assert tr.tensor_flags[63] == W.FLAG_REQUIRED
    w = W.make_config("chain32")
    assert w.specs["budget"].tolist()[:4] == [math.ceil(2 * math.sqrt(32)), 16, 32, 64]


def test_resnet_and_transformer_shapes():
    w = W.make_config("resnet50blk")
    _valid(w.traces[0])
    assert w.traces[0].n_ops == 604 and w.n_sims == 1536
    assert sorted(set(w.specs["heuristic"].tolist())) == [0, 1, 2, 3, 4, 5]
    w = W.make_config("transformer12")
    tr = w.traces[0]
    _valid(tr)
    assert tr.n_ops == 1108 and w.n_sims == 1536
    assert tr.op_cost[2] == 14496                  # QKV projection, FLOPs/1e6
    assert tr.tensor_size[2] == 8 * 512 * 3 * 768 * 2


def test_budgets_are_exact_integer_fractions():
    b = W.linear_budgets(1000, 10, 100, 4)
    assert b == [100, 400, 700, 1000]
    w = W.make_config("resnet50blk")
    bb = w.specs["budget"][:256]
    assert bb[-1] == w.peaks[0] and bb[0] == w.peaks[0] * 10 // 100


def test_treelstm_sizes():
    w = W.make_config("treelstm4096", n_trees=16)
    for tr in w.traces:
        _valid(tr)
        L = tr.meta["leaves"]
        assert 64 <= L <= 512
        assert tr.n_ops == 10 * (2 * L - 1) + 2
    assert w.n_sims == 16 * 8
    assert W.treelstm_trace(W.splitmix64(4 << 32)).digest() == w.traces[0].digest()


def test_random_dag_locality():
    tr = W.random_dag_trace(n_forward=3000)
    _valid(tr)
    F = 3000
    for o in range(1, F):
        ins = tr.inputs(o)
        assert 1 <= len(ins) <= 3 and (ins >= o - 64).all() and (ins < o).all()
    assert tr.n_ops == 2 * F


@pytest.mark.parametrize("seed", range(10))
def test_random_programs_valid(seed):
    _valid(W.random_program(seed, n_ops=40, n_const=5, backward=False))
    _valid(W.random_program(seed, n_ops=40, backward=True))


def test_log_peak_is_the_unlimited_replay_peak(oracle_lib):
    """The no-eviction memory profile that spaces log budgets equals the peak
    the oracle reaches with an unlimited budget (eager eviction of released
    storages, constants kept)."""
    logs = [W.random_log(s, n_steps=40 + 7 * s, n_const=s % 4) for s in range(30)] + [W.resnet_log(blocks=3)]
    specs = W.make_specs([(i, W.H_LRU, W.BUDGET_UNLIMITED, 0) for i in range(len(logs))])
    res = oracle_lib.run_log(logs, specs)
    assert [W.log_peak(L) for L in logs] == [int(v) for v in res["peak_memory"]]
    assert (res["n_evictions"] == 0).all() and (res["n_remats"] == 0).all()


def test_resnet_log_uses_the_instruction_kinds():
    L = W.resnet_log(blocks=4)
    kinds = set(int(k) for k in L.kind)
    assert kinds >= {W.LOG_MEMORY, W.LOG_ALIAS, W.LOG_CALL, W.LOG_MUTATE, W.LOG_CONSTANT, W.LOG_COPY,
                     W.LOG_RELEASE}
    assert L.digest() == W.resnet_log(blocks=4).digest()


def test_randdag100k_golden_matches_generator():
    """The stored oracle results of the full random-DAG workload belong to
    the trace and budgets the generator makes today."""
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "randdag100k_oracle.json")))
    w = W.make_config("randdag100k")
    assert w.traces[0].digest() == g["trace_sha256"]
    assert int(w.peaks[0]) == g["peak"] and w.n_sims == g["n_budgets"]
    pcts = []
    for s in g["sims"]:
        assert int(w.specs["budget"][s["index"]]) == s["budget"]
        assert int(w.specs["seed"][s["index"]]) == s["seed"]
        pcts.append(100 * s["budget"] / g["peak"])
    assert min(pcts) <= 5.01 and max(pcts) >= 99.99 and len(pcts) >= 8
