"""Benchmark of the batched DTR eviction-loop simulator on one MI355X.

A step is one pass of the whole hot path over one batch: every simulation of
the workload replayed end to end by ``dtr_sim_run`` (operator calls,
rematerializations, eviction scans, eager evictions, output condition).
Inputs are resident in HBM before the timed region (uploaded once by
``dtr_sim_create``).

Default workload: 4096 seeded TreeLSTM traces (64-512 leaves, hidden 256,
forward + backward), 8 budgets each from 20% to 100% of the trace's own peak,
heuristic h_DTR^eq: 32768 simulations.

Prints one JSON line.  ``value`` is simulated tensor ops per second (trace ops
plus rematerializations executed, summed over the batch, per second of GPU
time); eviction scores per second and the achieved fraction of HBM bandwidth
on the eviction-scoring reads (roofline) ride along.  ``cpu_baseline`` is the
plain CPU oracle timed on a bounded, deterministic sample of the same batch.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2006_09616_amd import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s

# Algorithmic bytes the scoring scan must read (canonical widths: id 4 B,
# size/last-access/cost 8 B each, state 1 B, set id 4 B, set cost 8 B).
#   every scored candidate: pool entry (id, size, c0, last access) 28 B
#                           + neighbourhood offsets 8 B            (h_DTR^eq, h_DTR)
#   every neighbour slot examined: id 4 B + state 1 B
#   every evicted neighbour (h_DTR^eq): set id 4 B + set running cost 8 B
#   every e* member (h_DTR): id 4 B + state 1 B + c0 8 B
PER_SCORE = {W.H_EQ: 36, W.H_DTR: 36, W.H_ESTAR: 36, W.H_LOCAL: 28, W.H_LRU: 12, W.H_SIZE: 12, W.H_RAND: 4}


def scan_bytes(specs, res) -> int:
    total = 0
    for h, per in PER_SCORE.items():
        m = specs["heuristic"] == h
        if not m.any():
            continue
        total += per * int(res["n_scores"][m].sum())
        if h == W.H_EQ:
            total += 5 * int(res["n_adj_visits"][m].sum()) + 12 * int(res["n_nbr_visits"][m].sum())
        elif h in (W.H_DTR, W.H_ESTAR):
            total += 5 * int(res["n_adj_visits"][m].sum()) + 13 * int(res["n_nbr_visits"][m].sum())
    return total


# HBM traffic of the replay kernel, measured with rocprofv3 counter passes
# (FETCH_SIZE, WRITE_SIZE) and scaled by the same counters on a plain device
# copy of known size; valid only for the kernel sources it was measured on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "replay_kernel_eq_treelstm4096_traffic.md")
# (the host library too: its dispatch order decides which simulations share the caches)
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2006_09616_amd", "csrc", f) for f in ("replay.hip", "layout.h", "dtr_sim.cpp")]


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per launch from the committed counter summary, or None when
    there is none for this workload or the kernel changed since it was taken."""
    if workload != "treelstm4096" or not os.path.exists(TRAFFIC_FILE):
        return None
    text = open(TRAFFIC_FILE).read()
    m_b = re.search(r"^traffic_bytes_per_launch:\s*(\d+)", text, re.M)
    m_h = re.search(r"^kernel_source_sha256:\s*([0-9a-f]{64})", text, re.M)
    if not m_b or not m_h or m_h.group(1) != kernel_source_digest():
        return None
    return int(m_b.group(1))


def copy_probe(mib: int):
    """A plain device-to-device copy of known size (counter calibration)."""
    import torch
    n = mib << 20
    x = torch.ones(n, dtype=torch.uint8, device="cuda:0")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "copies": 3}))


def _timed(traces, specs, steps: int):
    """Results and mean event-timed launch (ms) of one batch."""
    import torch
    from paper_2006_09616_amd import dtr as D
    sim = D.Simulator(traces, specs, device="cuda:0")
    sim.run()
    torch.cuda.synchronize()
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for i in range(steps):
        ev0[i].record(sim.stream)
        sim.run()
        ev1[i].record(sim.stream)
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in zip(ev0, ev1)) / steps
    res = sim.results()
    sim.close()
    return res, ms


def _variant_rows(traces, variants, steps: int, label: str):
    """Each variant (name -> specs) timed; the first is the reference for the
    total-cost ratios (simulations that finish under both), the OOM count
    and the speedup."""
    out, base = {}, None
    for name, specs in variants.items():
        res, ms = _timed(traces, specs, steps)
        ok = res["status"] == 0
        row = {"sims": int(len(specs)), "launch_ms": ms, "oom_rate": float(np.mean(res["status"] == 1)),
               "scores": int(res["n_scores"].sum()), "ops": int(res["n_executed_ops"].sum()),
               "ops_per_s": int(res["n_executed_ops"].sum()) / (ms / 1e3)}
        if base is None:
            base = (res, ms)
        else:
            both = ok & (base[0]["status"] == 0)
            ratio = res["total_cost"][both] / base[0]["total_cost"][both]
            row.update(speedup=base[1] / ms, cost_ratio_mean=float(ratio.mean()) if both.any() else None,
                       cost_ratio_max=float(ratio.max()) if both.any() else None,
                       scores_vs_first=row["scores"] / max(1, int(base[0]["n_scores"].sum())),
                       newly_oom=int(((res["status"] == 1) & (base[0]["status"] == 0)).sum()))
        out[name] = row
        print(f"[bench] {label} {name}: {ms:.1f} ms, oom {row['oom_rate']:.4f}", file=sys.stderr, flush=True)
    return out


def search_study(wl, steps: int):
    """The prototype's search approximations (ignore small candidates, sample
    sqrt(n) of the pool; Appendix E) against exact search on the same batch:
    OOM rate, total cost relative to exact search where both finish, scores
    searched, and launch time."""
    variants = {}
    for name, flags in {"exact": 0, "ignore_small": W.SEARCH_IGNORE_SMALL, "sample": W.SEARCH_SAMPLE,
                        "ignore_small+sample": W.SEARCH_IGNORE_SMALL | W.SEARCH_SAMPLE}.items():
        specs = wl.specs.copy()
        specs["search"] = flags
        variants[name] = specs
    return _variant_rows(wl.traces, variants, steps, "search study")


def _union_find(h: int) -> bool:
    return h == W.H_EQ or (h >= W.H_FAMILY and (h - W.H_FAMILY) >> 2 == W.C_EQCLASS)


def policy_study(wl, steps: int):
    """The deallocation policies (Section 2 and Appendix C.5: eager eviction at
    release, ignoring releases, banishing) on the same simulations, eager
    first.  Union-find heuristics take no banishing, so their simulations are
    left out of every variant."""
    keep = np.array([not _union_find(int(h)) for h in wl.specs["heuristic"]])
    if not keep.any():
        sys.exit("--study policy needs simulations whose heuristic is not a union-find one")
    variants = {}
    for name, pol in {"eager": W.POLICY_EAGER, "ignore": W.POLICY_IGNORE, "banish": W.POLICY_BANISH}.items():
        specs = wl.specs[keep].copy()
        specs["policy"] = pol
        variants[name] = specs
    return _variant_rows(wl.traces, variants, steps, "policy study")


def family_study(wl, steps: int):
    """h_MSPS and the ablation family h'(s, m, c) = c / (m^[m] s^[s]) for every
    cost measure c (e*, union-find neighbourhood, local, none; Section 4.1,
    Appendix A.3) on the budgets of the batch's h_DTR simulations (all
    simulations if it has none), h_DTR first."""
    rows = wl.specs[wl.specs["heuristic"] == W.H_DTR]
    if len(rows) == 0:
        rows = wl.specs
    variants = {}
    names = {W.C_ESTAR: "e*", W.C_EQCLASS: "eq", W.C_LOCAL: "local", W.C_NONE: "none"}
    for name, h in [("h_DTR", W.H_DTR), ("h_MSPS", W.H_MSPS)] + [
            (f"h'(c={names[c]},s={st},m={m})", W.h_family(c, st, m))
            for c in (W.C_ESTAR, W.C_EQCLASS, W.C_LOCAL, W.C_NONE) for st in (1, 0) for m in (1, 0)]:
        specs = rows.copy()
        specs["heuristic"] = h
        specs["policy"] = W.POLICY_EAGER
        variants[name] = specs
    return _variant_rows(wl.traces, variants, steps, "family study")


WORKLOADS = {
    "treelstm4096": lambda: W.make_config("treelstm4096"),
    "resnet50blk": lambda: W.make_config("resnet50blk"),
    "transformer12": lambda: W.make_config("transformer12"),
    "chain32": lambda: W.make_config("chain32"),
    "resnet50log": lambda: W.make_config("resnet50log"),
    "randdag100k": lambda: W.make_config("randdag100k"),
    # the random-DAG recipe at 10k forward ops (20k ops), 1024 budgets 5-100%, h_DTR
    "randdag10k": lambda: W.config_random_dag(n_forward=10_000, n_budgets=1024),
    # the full-size random DAG at its five stored budgets from 48% to 100%
    "randdag100k-stored": lambda: randdag_stored(),
}


def is_log(wl) -> bool:
    """Operator-log workloads replay through dtr_log_create (Appendix C.6)."""
    return isinstance(wl.traces[0], W.Log)


def ordinal(n: int) -> str:
    """1st, 2nd, 3rd, 4th, ..., 11th, 12th, 13th, ..., 21st, 61st."""
    suffix = "th" if 10 <= n % 100 <= 20 else {1: "st", 2: "nd", 3: "rd"}.get(n % 10, "th")
    return f"{n}{suffix}"


def cpu_baseline(wl, gpu_res, sample_every: int, threads: int, single_every: int = 29):
    """The oracle, as it stands, on every sample_every-th simulation, and its
    single-core rate on every single_every-th of those (29 keeps the stride
    coprime to the 8 budgets per tree whenever sample_every is)."""
    from oracle import oracle as O
    run = O.run_log if is_log(wl) else O.run
    idx = np.arange(0, wl.n_sims, sample_every)
    specs = wl.specs[idx]
    t0 = time.perf_counter()
    ref = run(wl.traces, specs, threads=threads)
    dt = time.perf_counter() - t0
    ops = int(ref["n_executed_ops"].sum())
    scores = int(ref["n_scores"].sum())
    match = sum(all(int(gpu_res[f][i]) == int(ref[f][k]) for f in O.RESULT_FIELDS)
                for k, i in enumerate(idx))
    out = dict(value=ops / dt, unit="simulated tensor ops/s", cores=threads, nproc=os.cpu_count(), kind="oracle",
               sample=f"every {ordinal(sample_every)} simulation ({len(idx)} of {wl.n_sims}), "
                      f"{dt:.2f} s wall on {threads} threads",
               scores_per_s=scores / dt, parity_sample=f"{match}/{len(idx)}")
    idx1 = idx[::single_every]
    t0 = time.perf_counter()
    ref1 = run(wl.traces, wl.specs[idx1], threads=1)
    dt1 = max(time.perf_counter() - t0, 1e-9)
    out["single_thread"] = dict(value=int(ref1["n_executed_ops"].sum()) / dt1, unit="simulated tensor ops/s",
                                sample=f"every {ordinal(sample_every * single_every)} simulation ({len(idx1)} of "
                                       f"{wl.n_sims}), {dt1:.2f} s on 1 thread")
    return out


RANDDAG_GOLDEN = os.path.join(ROOT, "tests", "golden", "randdag100k_oracle.json")


def sub_workloads():
    """The other benchmark configurations, each measured in the same run:
    the Appendix A chain, the ResNet and transformer batches in full, and the
    full-size random DAG (200k ops, h_DTR) at its stored oracle budgets from
    48% to 100% of the peak (the lower budgets take the GPU several minutes
    per simulation; their stored results are checked separately)."""
    out = [W.make_config("chain32"), W.make_config("resnet50blk"), W.make_config("transformer12")]
    out.append(randdag_stored())
    return out


def randdag_stored(lo_index: int = 460):
    """The full-size random DAG at its stored oracle budgets from index
    lo_index of 1024 up (460: 48%-100% of the peak), with those results."""
    g = json.load(open(RANDDAG_GOLDEN))
    full = W.make_config("randdag100k")
    rows = [r for r in g["sims"] if r["index"] >= lo_index]
    pick = np.array([r["index"] for r in rows])
    sub = W.Workload("randdag100k", full.traces, full.specs[pick], full.peaks,
                     f"random DAG 100k fwd ops, h_DTR, budget indices {pick.tolist()} of 1024 (48%-100% of peak)")
    sub.golden = rows
    return sub


def measure_sub(wl, steps: int, threads: int) -> dict:
    """One configuration: event-timed launches, throughput, algorithmic
    scan bytes, and the oracle on the host cores (run in a thread while the
    GPU works): on every simulation for the small batches, on the 90% budget
    for the random DAG, whose other stored results serve as parity."""
    import threading
    import torch
    from oracle import oracle as O
    from paper_2006_09616_amd import dtr as D
    golden = getattr(wl, "golden", None)
    cpu_idx = np.array([k for k, r in enumerate(golden) if r["index"] == 921]) if golden else np.arange(wl.n_sims)
    cpu = {}

    def oracle_leg():
        t0 = time.perf_counter()
        cpu["ref"] = O.run(wl.traces, wl.specs[cpu_idx], threads=threads)
        cpu["dt"] = time.perf_counter() - t0

    th = threading.Thread(target=oracle_leg)
    th.start()
    sim = D.Simulator(wl.traces, wl.specs, device="cuda:0")
    if not golden:
        sim.run()
        torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(sim.stream)
        sim.run()
        b.record(sim.stream)
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in ev) / steps
    res = sim.results()
    sim.close()
    th.join()
    ref, dt = cpu["ref"], cpu["dt"]
    cpu_match = sum(all(int(res[f][i]) == int(ref[f][k]) for f in O.RESULT_FIELDS) for k, i in enumerate(cpu_idx))
    if golden:
        parity = sum(all(int(res[f][k]) == v for f, v in r["result"].items()) for k, r in enumerate(golden))
        parity_of = "stored oracle results"
    else:
        parity, parity_of = cpu_match, "oracle in this run"
    ops, scores = int(res["n_executed_ops"].sum()), int(res["n_scores"].sum())
    nbytes = scan_bytes(wl.specs, res)
    achieved = nbytes / (ms / 1e3) / 1e9
    print(f"[bench] {wl.name}: {ms:.1f} ms per launch, parity {parity}/{wl.n_sims}, oracle {dt:.2f} s",
          file=sys.stderr, flush=True)
    return {"workload": wl.name, "description": wl.description, "n_sims": wl.n_sims, "launch_ms": ms,
            "launches": steps, "ops_per_s": ops / (ms / 1e3), "scores_per_s": scores / (ms / 1e3),
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBS, "algorithmic_bytes_per_launch": nbytes},
            "parity": f"{parity}/{wl.n_sims} bit-exact against the {parity_of}",
            "cpu_baseline": {"value": int(ref["n_executed_ops"].sum()) / dt, "unit": "simulated tensor ops/s",
                             "cores": threads, "nproc": os.cpu_count(), "kind": "oracle",
                             "sample": f"{len(cpu_idx)} of {wl.n_sims} simulations, {dt:.2f} s wall",
                             "parity_sample": f"{cpu_match}/{len(cpu_idx)}"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="treelstm4096", choices=sorted(WORKLOADS))
    ap.add_argument("--slots", type=int, default=0)
    ap.add_argument("--cpu-sample", type=int, default=61,
                    help="oracle on every k-th simulation (0: skip); 61 is coprime to the 8 budgets per tree")
    ap.add_argument("--cpu-threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--search-study", action="store_true",
                    help="only compare the search approximations with exact search on the workload")
    ap.add_argument("--study", choices=("search", "policy", "family"), default=None,
                    help="only compare variants of the workload's simulations: search approximations, "
                         "deallocation policies, or h_MSPS and the h'(s, m, c) family")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other configurations (chain, ResNet, transformer, random DAG)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU (--gpus 1): simulations are independent and would shard "
              "across GPUs by simulation with no exchange, which is not run here.", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe > 0:
        copy_probe(args.copy_probe)
        return

    import torch
    from paper_2006_09616_amd import dtr as D

    D.lib()
    t0 = time.perf_counter()
    wl = WORKLOADS[args.workload]()
    gen_s = time.perf_counter() - t0
    print(f"[bench] workload {wl.name}: {len(wl.traces)} traces, {wl.n_sims} sims, generated in {gen_s:.1f}s",
          file=sys.stderr, flush=True)
    study = "search" if args.search_study else args.study
    if study and is_log(wl):
        sys.exit("the studies run on trace workloads")
    if study:
        torch.cuda.set_device(0)
        fn = {"search": search_study, "policy": policy_study, "family": family_study}[study]
        print(json.dumps({f"{study}_study": fn(wl, args.steps), "workload": wl.name,
                          "n_sims": wl.n_sims, "n_gpus": 1}))
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log = is_log(wl)
    sim = D.Simulator(None if log else wl.traces, wl.specs, device="cuda:0", slots=args.slots,
                      logs=wl.traces if log else None)
    stream = sim.stream
    def wait(label):
        # a launch that lasts minutes reports the operations its walk
        # simulations have executed so far (dtr_sim_progress) while it runs
        t = time.perf_counter()
        while not log and not sim.done():
            time.sleep(0.05 if time.perf_counter() - t < 30 else 20)
            if time.perf_counter() - t >= 30:
                print(f"[bench] {label}: {time.perf_counter() - t:.0f} s, {sim.progress()} operations executed",
                      file=sys.stderr, flush=True)
        torch.cuda.synchronize()

    for i in range(args.warmup):
        sim.run()
        wait(f"warmup {i + 1}")
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        sim.run()
        ends[i].record(stream)
    wait("timed steps")
    wall = time.perf_counter() - w0
    launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    res = sim.results()
    avg_s = sum(launch_ms) / len(launch_ms) / 1e3
    ops = int(res["n_executed_ops"].sum())
    scores = int(res["n_scores"].sum())
    nbytes = scan_bytes(wl.specs, res)
    achieved = nbytes / avg_s / 1e9
    print(f"[bench] {args.steps} steps, kernel avg {avg_s * 1e3:.2f} ms, wall {wall:.3f}s",
          file=sys.stderr, flush=True)

    golden = None
    if getattr(wl, "golden", None):
        # a subset of the random-DAG batch, with its stored oracle results
        ok = sum(all(int(res[f][k]) == v for f, v in r["result"].items()) for k, r in enumerate(wl.golden))
        golden = f"{ok}/{len(wl.golden)} bit-exact against the stored oracle results"
    elif wl.name.startswith("randdag") and os.path.exists(RANDDAG_GOLDEN):
        # the stored oracle results at 9 of the batch's budgets
        g = json.load(open(RANDDAG_GOLDEN))
        if g["trace_sha256"] == wl.traces[0].digest() and g["n_budgets"] == wl.n_sims:
            ok = sum(all(int(res[f][r["index"]]) == v for f, v in r["result"].items()) for r in g["sims"])
            golden = f"{ok}/{len(g['sims'])} bit-exact against the stored oracle results"
    if golden:
        print(f"[bench] stored oracle results: {golden}", file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_sample > 0:
        cpu = cpu_baseline(wl, res, args.cpu_sample, args.cpu_threads)
        print(f"[bench] cpu baseline: {cpu['sample']}, parity {cpu['parity_sample']}",
              file=sys.stderr, flush=True)

    configs = None
    if not args.no_configs and args.workload == "treelstm4096":
        configs = [measure_sub(w, 1 if getattr(w, "golden", None) else 3, args.cpu_threads) for w in sub_workloads()]

    status = np.bincount(res["status"], minlength=4).tolist()
    traffic = measured_traffic(wl.name)
    # `achieved` and `frac` are algorithmic (the method's bytes per launch over
    # the launch time); the HBM traffic the counters saw, when its summary
    # matches these kernel sources, gives measured_gbs and measured_frac
    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                "kernel": "log_kernel" if log else "replay_kernel", "algorithmic_bytes_per_launch": nbytes,
                "avg_launch_ms": avg_s * 1e3}
    if traffic is not None:
        roofline["measured_gbs"] = traffic / avg_s / 1e9
        roofline["measured_frac"] = traffic / avg_s / 1e9 / HBM_PEAK_GBS
    out = {
        "metric": "simulated tensor ops/sec + eviction scores/sec (1 GPU), % peak HBM BW",
        "value": ops / avg_s,
        "unit": "simulated tensor ops/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "n_sims": wl.n_sims,
                   "n_traces": len(wl.traces), "ops_per_step": ops, "scores_per_step": scores,
                   "status_counts": {"ok": status[0], "oom": status[1], "clock": status[2],
                                     "capacity": status[3]},
                   "trace_sha256": wl.digest()[:16]},
        "eviction_scores_per_s": scores / avg_s,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "configs": configs,
        **({"parity_stored": golden} if golden else {}),
    }
    print(json.dumps(out))
    sim.close()


if __name__ == "__main__":
    main()
