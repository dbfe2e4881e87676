"""Host-side logic of bench.py (no GPU): the one-GPU rule, the algorithmic
scan-byte count behind the roofline figure, and the gating of the measured
HBM traffic on the kernel sources it was measured with."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2006_09616_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_scan_bytes_counts_what_the_scores_read():
    specs = W.make_specs([(0, W.H_EQ, 10, 0), (0, W.H_EQ, 20, 0), (0, W.H_DTR, 10, 0), (0, W.H_LRU, 10, 0),
                          (0, W.H_RAND, 10, 0)])
    res = np.zeros(len(specs), dtype=[("n_scores", "i8"), ("n_adj_visits", "i8"), ("n_nbr_visits", "i8")])
    res["n_scores"] = [100, 10, 7, 1000, 50]
    res["n_adj_visits"] = [400, 40, 30, 0, 0]
    res["n_nbr_visits"] = [90, 9, 11, 0, 0]
    # h_DTR^eq: 36 per score + 5 per neighbour slot + 12 per evicted neighbour
    eq = 36 * 110 + 5 * 440 + 12 * 99
    # h_DTR: 36 per score + 5 per neighbour slot + 13 per e* member
    dtr = 36 * 7 + 5 * 30 + 13 * 11
    assert bench.scan_bytes(specs, res) == eq + dtr + 12 * 1000 + 4 * 50


def test_measured_traffic_is_gated_on_the_kernel_sources(monkeypatch):
    text = open(bench.TRAFFIC_FILE).read()
    recorded = int(text.split("traffic_bytes_per_launch:")[1].split()[0])
    assert bench.measured_traffic("resnet50blk") is None
    if bench.kernel_source_digest() in text:
        assert bench.measured_traffic("treelstm4096") == recorded
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.measured_traffic("treelstm4096") is None


def test_union_find_heuristics_are_recognised():
    uf = [h for h in list(range(8)) + list(range(16, 32)) if bench._union_find(h)]
    assert uf == [W.H_EQ] + [W.h_family(W.C_EQCLASS, s, m) for s in (0, 1) for m in (0, 1)]


def test_cpu_baseline_reports_both_rates_and_parity(oracle_lib):
    wl = W.make_config("chain32")
    ref = oracle_lib.run(wl.traces, wl.specs, threads=1)
    cpu = bench.cpu_baseline(wl, ref, 1, 2, single_every=2)
    assert cpu["kind"] == "oracle" and cpu["cores"] == 2
    assert cpu["parity_sample"] == f"{wl.n_sims}/{wl.n_sims}"
    assert cpu["value"] > 0 and cpu["single_thread"]["value"] > 0
    assert "1 thread" in cpu["single_thread"]["sample"]
    # a planted difference in the GPU side's results is counted
    bad = ref.copy()
    bad["total_cost"][0] += 1
    assert bench.cpu_baseline(wl, bad, 1, 2)["parity_sample"] == f"{wl.n_sims - 1}/{wl.n_sims}"


def test_ordinals():
    assert [bench.ordinal(n) for n in (1, 2, 3, 4, 11, 12, 13, 21, 61, 111, 1769)] == \
        ["1st", "2nd", "3rd", "4th", "11th", "12th", "13th", "21st", "61st", "111th", "1769th"]
