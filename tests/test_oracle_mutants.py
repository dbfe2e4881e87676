"""Mutation check of the oracle's pins (CPU only).

Each entry below plants one plausible mistake in a copy of the oracle source
(a dropped term, a wrong sign, index or bound, a transposed operand, a step
skipped), builds the copy with gcc, and runs the oracle's pin suites against
that build in a subprocess.  Every mutant must make a pin fail; the
unmutated copy, built and run the same way, must pass.  A mistake that no pin
notices would make the pins a restatement of the oracle rather than a check
of it.

The mistakes are taken against what the paper fixes: the greedy loop of
Section 2 and Appendix C.4 (locking, rematerialization, allocation, eviction,
the clock and its guard, the output condition), the scores of Section 4.1 and
Appendix C.3 (staleness, size, e*, e_R, the union-find relaxation and its
split approximation of Appendix C.2), the ablation family of Appendix D, the
deallocation policies of Appendix C.5, the search approximations of
Appendix E and the log semantics of Appendix C.6.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "dtr_oracle.c")
PIN_SUITES = ["tests/test_oracle_pins.py", "tests/test_log_pins.py"]

# (what the mistake is, text in the oracle source, replacement)
MUTANTS = [
    ("e* without its descendant half (Appendix C.2)",
     "if (s->state[c] != ST_EVICTED || s->mark[c] == s->epoch) continue;",
     "if (1) continue;"),
    ("e_R adds the cost of the tensor it came from instead of the parent's",
     "            sum += c0_of(s, p);\n",
     "            sum += c0_of(s, u);\n"),
    ("ties broken towards the larger id",
     "return ia < ib;",
     "return ia > ib;"),
    ("score comparison with its cross products transposed",
     "u128 l = (u128)na * db, r = (u128)nb * da;",
     "u128 l = (u128)na * da, r = (u128)nb * db;"),
    ("staleness one larger than clock minus last access",
     "int64_t stale = s->clock - s->last_access[x];",
     "int64_t stale = s->clock - s->last_access[x] + 1;"),
    ("h_DTR without the size term in its denominator",
     "        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;\n"
     "        s->r[R_NBR_VISITS] += cnt;\n"
     "        s->r[R_ADJ_VISITS] += degree(s, x);\n"
     "        break;\n"
     "    case OH_ESTAR:",
     "        *D = (u128)(uint64_t)stale;\n"
     "        s->r[R_NBR_VISITS] += cnt;\n"
     "        s->r[R_ADJ_VISITS] += degree(s, x);\n"
     "        break;\n"
     "    case OH_ESTAR:"),
    ("h_MSPS scored with the whole e* instead of the evicted ancestors (Section 4.1)",
     "*N = (uint64_t)(c0 + ancestors_cost(s, x, &cnt));",
     "*N = (uint64_t)(c0 + estar_cost(s, x, &cnt));"),
    ("ablation family with the size and staleness switches swapped (Appendix D)",
     "((h & 1) ? m : 1) * (u128)(uint64_t)((h & 2) ? stale : 1)",
     "((h & 2) ? m : 1) * (u128)(uint64_t)((h & 1) ? stale : 1)"),
    ("union-find neighbourhood counting a shared set once per neighbour",
     "if (s->uf_mark[r] == s->epoch) continue;",
     "if (0) continue;"),
    ("split approximation not subtracting the rematerialized tensor's cost",
     "s->uf_cost[r] -= s->g->c0[t];",
     "s->uf_cost[r] -= 0;"),
    ("eviction not adding the tensor's cost to its set",
     "s->uf_cost[r] += c0_of(s, v);",
     ";"),
    ("eviction not merging with evicted children",
     "if (s->state[c] == ST_EVICTED) r = uf_union(s, r, s->node_of[c]);",
     ";"),
    ("union dropping the absorbed set's cost",
     "s->uf_cost[a] += s->uf_cost[b];",
     ";"),
    ("output tensor's last access not stamped",
     "    s->last_access[t] = s->clock;\n    int64_t c = tr->op_cost[o];",
     "    int64_t c = tr->op_cost[o];"),
    ("inputs' last access not stamped",
     "        s->last_access[tr->op_inputs[e]] = s->clock;\n",
     "        ;\n"),
    ("peak not updated after an operator's output is allocated",
     "    s->memory += tr->tensor_size[t];\n    if (s->memory > s->peak) s->peak = s->memory;",
     "    s->memory += tr->tensor_size[t];"),
    ("evicting while memory plus the request reaches the budget (not exceeds it)",
     "while (s->memory + size > s->budget)",
     "while (s->memory + size >= s->budget)"),
    ("clock guard tripping only beyond 2^40 instead of at it",
     "    if (s->clock >= CLOCK_LIMIT) { s->r[R_STATUS] = OS_CLOCK_OVERFLOW; s->stopped = OS_CLOCK_OVERFLOW; }",
     "    if (s->clock > CLOCK_LIMIT) { s->r[R_STATUS] = OS_CLOCK_OVERFLOW; s->stopped = OS_CLOCK_OVERFLOW; }"),
    ("failed operator reported one past the one that failed",
     "    if (s->stopped == OS_OOM || s->stopped == OS_CLOCK_OVERFLOW) s->r[R_FAILED_OP] = s->cur_op;\n"
     "    s->r[R_PEAK] = s->peak;\n    s->r[R_FINAL_MEM] = s->memory;\n}\n\nstatic int run_one(",
     "    if (s->stopped == OS_OOM || s->stopped == OS_CLOCK_OVERFLOW) s->r[R_FAILED_OP] = s->cur_op + 1;\n"
     "    s->r[R_PEAK] = s->peak;\n    s->r[R_FINAL_MEM] = s->memory;\n}\n\nstatic int run_one("),
    ("tensors released after their first reader instead of their last",
     "if (last[u] < o) last[u] = o;",
     "if (last[u] < 0) last[u] = o;"),
    ("output condition skipped (required outputs not brought back)",
     "        if (!(tr->tensor_flags[t] & O_FLAG_REQUIRED)) continue;\n        lock(s, t);",
     "        continue;\n        lock(s, t);"),
    ("scores searched counted one short per decision",
     "s->r[R_SCORES] += count;",
     "s->r[R_SCORES] += count - 1;"),
    ("h_DTR's neighbourhood visits counted one too many per score",
     "        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;\n"
     "        s->r[R_NBR_VISITS] += cnt;\n",
     "        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;\n"
     "        s->r[R_NBR_VISITS] += cnt + 1;\n"),
    ("rematerialization cost not accumulated",
     "if (remat) { s->r[R_REMATS]++; s->r[R_REMAT_COST] += c; }\n    else s->r[R_BASE_COST] += c;\n    s->memory += tr->tensor_size[t];",
     "if (remat) { s->r[R_REMATS]++; }\n    else s->r[R_BASE_COST] += c;\n    s->memory += tr->tensor_size[t];"),
    ("sampling keeping floor(sqrt(n)) + 1 candidates instead of ceil(sqrt(n)) (Appendix E)",
     "while (r * r < n) r++;",
     "while (r * r <= n) r++;"),
    ("ignore-small threshold at 10% of the mean size instead of 1% (Appendix E)",
     "(u128)100 * (u128)(uint64_t)s->tr->tensor_size[x]",
     "(u128)10 * (u128)(uint64_t)s->tr->tensor_size[x]"),
    ("banishing leaving a banished tensor's children evictable (Appendix C.4)",
     "if (s->state[g->ch[e]] == ST_RESIDENT) s->pinned[g->ch[e]] = 1;",
     ";"),
    ("log: a view allocating its storage again (Appendix C.6 ALIAS)",
     "if (!L->t_alias.v[L->outs.v[e]]) need += L->s_size.v[L->t_storage.v[L->outs.v[e]]];",
     "need += L->s_size.v[L->t_storage.v[L->outs.v[e]]];"),
    ("log: a storage's cost overwritten by each operator writing it, not summed",
     "if (!L->s_const.v[st]) s->dc0[st] += L->op_cost.v[o];",
     "if (!L->s_const.v[st]) s->dc0[st] = L->op_cost.v[o];"),
    ("log: split approximation not subtracting the storage's cost",
     "s->uf_cost[r] -= c0_of(s, st);",
     "s->uf_cost[r] -= 0;"),
    ("log: inputs' last access not stamped",
     "    for (int64_t e = ib; e < ie; e++) s->last_access[L->t_storage.v[L->ins.v[e]]] = s->clock;\n",
     ""),
]


def _build(src_text: str, out: str) -> None:
    c = out[:-3] + ".c"
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", out, c])


def _run_pins(lib: str) -> tuple[int, str]:
    env = dict(os.environ, DTR_ORACLE_LIB=lib, OMP_NUM_THREADS="1")
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           "--timeout", "300", *PIN_SUITES]
    p = subprocess.run(cmd, cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    return p.returncode, p.stdout


def test_every_planted_mistake_fails_a_pin(tmp_path):
    with open(SRC) as f:
        src = f.read()
    jobs = [("unmutated", src)]
    for name, old, new in MUTANTS:
        assert old in src, f"mutation target gone from the oracle source: {name}"
        jobs.append((name, src.replace(old, new)))
    libs = []
    for k, (name, text) in enumerate(jobs):
        lib = str(tmp_path / f"mutant{k}.so")
        _build(text, lib)
        libs.append(lib)
    workers = max(1, min(8, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as ex:
        outs = list(ex.map(_run_pins, libs))
    rc0, log0 = outs[0]
    assert rc0 == 0, "the unmutated oracle must pass its pins:\n" + log0[-2000:]
    survivors, crashed = [], []
    for (name, _), (rc, log) in zip(jobs[1:], outs[1:]):
        # 1: a test failed; anything else (a crash, a collection error) is not
        # a pin catching the mistake
        if rc == 0:
            survivors.append(name)
        elif rc != 1:
            crashed.append(f"{name} (exit {rc}): {log[-400:]}")
    assert not survivors, "mistakes no pin notices: " + "; ".join(survivors)
    assert not crashed, "mutants that did not fail a pin cleanly: " + "; ".join(crashed)
