"""Per-simulation cycle profile of the trace kernels (a developer tool).

The library built with -DDTR_PROFILE (libdtrsim_prof.so beside the product
library; the product build carries no timers) records, per simulation, the
cycles of the whole replay, of its eviction scans and of each phase (evict,
execute, unlock, lock, release, resume, output, descend).  This runs chosen
simulations of a named workload alone, then (with --batch) the whole batch,
and prints cycles per executed operation and the distribution of simulation
times over the batch.  Build the profile library first:

    python -c "from paper_2006_09616_amd import build; build.build(profile=True)"
    python -m paper_2006_09616_amd.profile --workload treelstm4096 --sims 11080,5104 --batch
"""
from __future__ import annotations

import argparse
import ctypes as C
import os
import time

import numpy as np

from . import build as B
from . import dtr as D
from . import workloads as W

PHASES = ["evict", "execute", "unlock", "lock", "release", "resume", "output", "descend"]
CLOCK_HZ = 2.4e9          # the cycle counter's rate (shader clock)


def phase_line(label: str, prof: np.ndarray, ops: int) -> str:
    ops = max(1, int(ops))
    return (f"{label}: ops {ops} cycles/op {prof[0] / ops:.0f} scan {prof[1] / ops:.0f} "
            f"rounds/op {prof[3] / ops:.2f} | " +
            "  ".join(f"{n} {prof[8 + j] / ops:.0f}" for j, n in enumerate(PHASES)))


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="treelstm4096", choices=["treelstm4096", "resnet50blk", "transformer12"])
    ap.add_argument("--sims", default="", help="comma-separated simulation indices to run alone")
    ap.add_argument("--batch", action="store_true", help="also run the whole batch")
    args = ap.parse_args()
    if not os.path.exists(B.OUT_PROFILE):
        raise SystemExit(f"{B.OUT_PROFILE} is missing: build it with build.build(profile=True)")
    D.LIB_PATH = B.OUT_PROFILE
    import torch
    L = D.lib()
    L.dtr_sim_profile.argtypes = [C.c_void_p, C.c_void_p, C.c_int32]
    L.dtr_sim_profile.restype = C.c_int
    wl = W.make_config(args.workload)
    print(f"[profile] {wl.name}: {wl.n_sims} simulations", flush=True)
    for k in [int(x) for x in args.sims.split(",") if x]:
        one = wl.specs[k:k + 1].copy()
        tr = [wl.traces[int(one["trace"][0])]]
        one["trace"] = 0
        sim = D.Simulator(tr, one, device="cuda:0")
        sim.run()
        torch.cuda.synchronize()
        t = time.time()
        sim.run()
        torch.cuda.synchronize()
        dt = time.time() - t
        res = sim.results()
        prof = np.zeros((1, 16), np.int64)
        assert L.dtr_sim_profile(C.c_void_p(sim.handle), prof.ctypes.data, 1) == 0
        print(phase_line(f"sim {k} alone ({dt * 1e3:.0f} ms)", prof[0], res["n_executed_ops"][0]), flush=True)
        sim.close()
    if args.batch:
        sim = D.Simulator(wl.traces, wl.specs, device="cuda:0")
        sim.run()
        torch.cuda.synchronize()
        t = time.time()
        sim.run()
        torch.cuda.synchronize()
        dt = time.time() - t
        res = sim.results()
        prof = np.zeros((wl.n_sims, 16), np.int64)
        assert L.dtr_sim_profile(C.c_void_p(sim.handle), prof.ctypes.data, wl.n_sims) == 0
        secs = prof[:, 0] / CLOCK_HZ
        order = np.argsort(-secs)
        print(f"[profile] batch launch {dt * 1e3:.0f} ms; simulation times: total {secs.sum():.1f} s, "
              f"heaviest {secs.max():.3f} s", flush=True)
        for q in (1, 2, 5, 10, 20, 50, 100, 500, 1000, 2000):
            if q <= len(order):
                print(f"  {q}th heaviest: {secs[order[q - 1]]:.3f} s", flush=True)
        for k in order[:5]:
            print(phase_line(f"sim {int(k)} in the batch", prof[k], res["n_executed_ops"][k]), flush=True)
        sim.close()


if __name__ == "__main__":
    main()
