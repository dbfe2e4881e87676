"""Writes randdag100k_oracle.json: CPU-oracle results of the full-size random-DAG
workload (100k forward ops + 100k backward ops, h_DTR with the exact evicted
neighbourhood e*) at budgets spanning 5% to 100% of the program's peak.

Every stored value comes from ``oracle/`` run on the seeded trace of
``workloads.config_random_dag`` (the input generator, no method arithmetic);
nothing here touches the GPU path.  The exact-e* oracle needs minutes to tens
of minutes per low-budget simulation, so the results are stored rather than
recomputed by the tests.

    python tests/golden/make_randdag100k_golden.py [--threads 8]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor, as_completed

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2006_09616_amd import workloads as W  # noqa: E402

OUT = os.path.join(HERE, "randdag100k_oracle.json")
# budget indices of the 1024-budget batch: 5%, ~10%, ~19%, ~34%, ~48%, ~62%,
# ~76%, ~90% and 100% of the peak
INDICES = [0, 51, 154, 307, 460, 614, 767, 921, 1023]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    w = W.make_config("randdag100k")
    tr = w.traces[0]
    rows = {}
    t_all = time.time()

    def one(k):
        t0 = time.time()
        r = O.run(w.traces, w.specs[[k]], threads=1)[0]
        return k, {f: int(r[f]) for f in O.RESULT_FIELDS}, time.time() - t0

    with ThreadPoolExecutor(max_workers=args.threads) as ex:
        futs = [ex.submit(one, k) for k in sorted(INDICES, key=lambda k: k)]
        for f in as_completed(futs):
            k, res, dt = f.result()
            rows[k] = dict(index=k, budget=int(w.specs["budget"][k]), seed=int(w.specs["seed"][k]),
                           oracle_seconds=round(dt, 1), result=res)
            print(f"budget index {k}: {dt:.1f} s, {res['n_executed_ops']} ops, "
                  f"{res['n_nbr_visits']} e* members", flush=True)
    doc = {
        "what": "oracle results of the random-DAG workload at sampled budgets of its 1024-budget batch",
        "recipe": "workloads.make_config('randdag100k'): seed 5, 100k forward ops reading 1-3 of the "
                  "previous 64 outputs, log-normal sizes (median 1 MiB, sigma 1.5), cost "
                  "max(1, size // 4096) x U{1..8}, reverse-order backward pass; h_DTR; budgets "
                  "linearly spaced from 5% to 100% of the no-eviction peak",
        "written_by": "tests/golden/make_randdag100k_golden.py (calls oracle/ only)",
        "trace_sha256": tr.digest(),
        "peak": int(w.peaks[0]),
        "n_budgets": int(w.n_sims),
        "wall_seconds": round(time.time() - t_all, 1),
        "sims": [rows[k] for k in sorted(rows)],
    }
    with open(OUT, "w") as fh:
        json.dump(doc, fh, indent=1)
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
