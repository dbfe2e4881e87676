"""Exhaustive search over DTR's eviction choices, and a small independent
Python rendering of the same state machine.

The machine follows the operator call of Section 2 and Appendix C.4: lock the
inputs, rematerialize evicted inputs (recursively, in listed order), allocate
the output (evicting while memory is insufficient), run the operator, unlock,
then release tensors whose last reader has run (eager eviction, ignoring the
release, or banishing, Appendix C.4/C.5), and at the end rematerialize and
lock the required outputs (Appendix C.6).
It is written as an explicit-stack machine so that a state at an eviction
decision is a hashable value; the only nondeterminism is *which* evictable
tensor is evicted.

``opt_cost`` explores every choice at every decision (memoised on the state)
and returns the minimum total cost, or None if every branch runs out of
memory.  Since a heuristic run is one branch of this search, every heuristic's
total cost is >= opt_cost, and if opt_cost is None every heuristic must
report out-of-memory.

``simulate`` takes the argmin of a heuristic score at each decision instead,
using Python integers and Fractions; it is used on small programs as a
second, independently written simulator.
"""
from __future__ import annotations

import sys
from fractions import Fraction

UNCOMPUTED, RESIDENT, EVICTED, BANISHED = 0, 1, 2, 3
EAGER, IGNORE, BANISH = 0, 1, 2
FLAG_CONSTANT, FLAG_REQUIRED = 1, 2
CLOCK_LIMIT = 1 << 40
MASK64 = (1 << 64) - 1


class Program:
    def __init__(self, trace):
        self.n = trace.n_tensors
        self.F = trace.n_ops
        self.size = [int(v) for v in trace.tensor_size]
        self.flags = [int(v) for v in trace.tensor_flags]
        self.out = [int(v) for v in trace.op_output]
        self.cost = [int(v) for v in trace.op_cost]
        off = [int(v) for v in trace.op_input_offsets]
        flat = [int(v) for v in trace.op_inputs]
        self.ins = [flat[off[o]:off[o + 1]] for o in range(self.F)]
        self.producer = [-1] * self.n
        for o, t in enumerate(self.out):
            self.producer[t] = o
        self.c0 = [self.cost[self.producer[t]] if self.producer[t] >= 0 else 0 for t in range(self.n)]
        self.parents = [self.ins[self.producer[t]] if self.producer[t] >= 0 else [] for t in range(self.n)]
        self.children = [[] for _ in range(self.n)]
        for o in range(self.F):
            for u in self.ins[o]:
                self.children[u].append(self.out[o])
        last = [-1] * self.n
        for o in range(self.F):
            last[self.out[o]] = max(last[self.out[o]], o)
            for u in self.ins[o]:
                last[u] = max(last[u], o)
        self.release = [[] for _ in range(self.F)]
        for t in range(self.n):
            if self.flags[t] & FLAG_REQUIRED or last[t] < 0:
                continue
            self.release[last[t]].append(t)
        self.required = [t for t in range(self.n) if self.flags[t] & FLAG_REQUIRED]


class Machine:
    """Explicit-stack DTR machine.  Frames: ['op', o, i], ['remat', u, i],
    ['out', k]; i == -1 means the inputs are not locked yet."""

    __slots__ = ("p", "budget", "frames", "state", "locks", "mem", "peak", "cost", "remat_cost",
                 "clock", "last", "done", "oom", "overflow", "n_evict", "n_eager", "n_remat",
                 "n_exec", "n_scores", "uf", "evict_no", "policy", "pinned", "pending")

    def __init__(self, prog: Program, budget: int, track_uf: bool = False, policy: int = EAGER):
        self.p = prog
        self.budget = budget
        self.policy = policy
        self.pinned = [False] * prog.n
        self.pending = [False] * prog.n
        self.state = [UNCOMPUTED] * prog.n
        self.locks = [0] * prog.n
        self.last = [0] * prog.n
        self.mem = 0
        for t in range(prog.n):
            if prog.flags[t] & FLAG_CONSTANT:
                self.state[t] = RESIDENT
                self.mem += prog.size[t]
        self.peak = self.mem
        self.cost = self.remat_cost = self.clock = 0
        self.done = self.oom = self.overflow = False
        self.n_evict = self.n_eager = self.n_remat = self.n_exec = self.n_scores = 0
        self.evict_no = 0
        self.uf = UnionFind() if track_uf else None
        self.frames = [["op", 0, -1]] if prog.F > 0 else [["out", 0]]
        if self.mem > budget:
            self.oom = True

    def copy(self):
        m = Machine.__new__(Machine)
        for k in Machine.__slots__:
            v = getattr(self, k)
            if k == "frames":
                v = [list(f) for f in v]
            elif isinstance(v, list):
                v = list(v)
            setattr(m, k, v)
        return m

    def key(self):
        return (tuple(tuple(f) for f in self.frames), tuple(self.state), tuple(self.locks),
                tuple(self.pinned), tuple(self.pending))

    def candidates(self):
        p = self.p
        return [x for x in range(p.n) if self.state[x] == RESIDENT and self.locks[x] == 0
                and not p.flags[x] & FLAG_CONSTANT and not self.pinned[x]]

    def evict(self, x, eager=False):
        self.state[x] = EVICTED
        self.mem -= self.p.size[x]
        if eager:
            self.n_eager += 1
        else:
            self.n_evict += 1
            self.evict_no += 1
        if self.uf is not None:
            self.uf.on_evict(x, self)

    def banish(self, t):
        """Permanent removal once no child is evicted and nothing holds t;
        resident children become pinned.  Else t waits for a child's remat."""
        p = self.p
        if self.locks[t] > 0 or any(self.state[c] == EVICTED for c in p.children[t]):
            self.pending[t] = True
            return
        self.pending[t] = False
        if self.state[t] == RESIDENT:
            self.mem -= p.size[t]
        self.state[t] = BANISHED
        self.n_eager += 1
        for c in p.children[t]:
            if self.state[c] == RESIDENT:
                self.pinned[c] = True

    def _frame_op(self, f):
        return f[1] if f[0] == "op" else self.p.producer[f[1]]

    def run(self):
        """Run deterministically until an eviction decision is needed
        (returns the candidate list), or the program ends / fails (returns None)."""
        p = self.p
        while not (self.done or self.oom or self.overflow):
            f = self.frames[-1]
            if f[0] == "out":
                k = f[1]
                if k == len(p.required):
                    self.done = True
                    break
                t = p.required[k]
                if f[-1] != "locked":
                    self.locks[t] += 1
                    f.append("locked")
                if self.state[t] == EVICTED:
                    self.frames.append(["remat", t, -1])
                else:
                    self.frames[-1] = ["out", k + 1]
                continue
            o = self._frame_op(f)
            ins = p.ins[o]
            if f[2] == -1:
                for u in ins:
                    assert self.state[u] != BANISHED
                    self.locks[u] += 1
                f[2] = 0
            if f[2] < len(ins):
                u = ins[f[2]]
                f[2] += 1
                if self.state[u] == EVICTED:
                    self.frames.append(["remat", u, -1])
                continue
            t = p.out[o]
            if self.mem + p.size[t] > self.budget:
                c = self.candidates()
                if not c:
                    self.oom = True
                    return None
                return c
            # execute
            for u in ins:
                self.last[u] = self.clock
            self.last[t] = self.clock
            self.clock += p.cost[o]
            self.cost += p.cost[o]
            self.n_exec += 1
            if f[0] == "remat":
                self.remat_cost += p.cost[o]
                self.n_remat += 1
            self.mem += p.size[t]
            self.peak = max(self.peak, self.mem)
            self.state[t] = RESIDENT
            if self.uf is not None:
                self.uf.on_materialize(t, f[0] == "remat", self)
            if self.clock >= CLOCK_LIMIT:
                self.overflow = True
                return None
            for u in ins:
                self.locks[u] -= 1
            self.frames.pop()
            if f[0] == "remat" and self.policy == BANISH:
                for u in ins:
                    if self.pending[u]:
                        self.banish(u)
            if f[0] == "op":
                for r in p.release[o]:
                    if self.policy == EAGER:
                        if self.state[r] == RESIDENT and self.locks[r] == 0 and not p.flags[r] & FLAG_CONSTANT \
                                and not self.pinned[r]:
                            self.evict(r, eager=True)
                    elif self.policy == BANISH:
                        self.banish(r)
                self.frames.append(["op", o + 1, -1] if o + 1 < p.F else ["out", 0])
        return None


def opt_cost(trace, budget: int):
    """Minimum total cost over every sequence of eviction choices (None if all OOM)."""
    prog = Program(trace)
    sys.setrecursionlimit(max(sys.getrecursionlimit(), 100000))
    memo = {}

    def solve(m, cands):
        key = m.key()
        if key in memo:
            return memo[key]
        best = None
        base = m.cost
        for x in cands:
            m2 = m.copy()
            m2.evict(x)
            c2 = m2.run()
            if m2.oom:
                continue
            if c2 is None:
                val = m2.cost - base
            else:
                sub = solve(m2, c2)
                if sub is None:
                    continue
                val = m2.cost - base + sub
            if best is None or val < best:
                best = val
        memo[key] = best
        return best

    m = Machine(prog, budget)
    if m.oom:
        return None
    c = m.run()
    if m.oom:
        return None
    if c is None:
        return m.cost
    sub = solve(m, c)
    return None if sub is None else m.cost + sub


class UnionFind:
    """Evicted components with the split approximation (Appendix C.2), kept
    as explicit member sets of (tensor, incarnation) nodes."""

    def __init__(self):
        self.node = {}          # tensor -> current node (tensor, incarnation)
        self.inc = {}
        self.comp = {}          # node -> component id
        self.members = {}       # component id -> set of nodes
        self.ccost = {}         # component id -> running cost
        self.next = 0

    def _fresh(self, t):
        self.inc[t] = self.inc.get(t, -1) + 1
        nd = (t, self.inc[t])
        cid = self.next
        self.next += 1
        self.node[t] = nd
        self.comp[nd] = cid
        self.members[cid] = {nd}
        self.ccost[cid] = 0

    def on_materialize(self, t, remat, m):
        if remat:
            self.ccost[self.comp[self.node[t]]] -= m.p.c0[t]
        self._fresh(t)

    def _merge(self, a, b):
        if a == b:
            return a
        for nd in self.members[b]:
            self.comp[nd] = a
        self.members[a] |= self.members.pop(b)
        self.ccost[a] += self.ccost.pop(b)
        return a

    def on_evict(self, v, m):
        a = self.comp[self.node[v]]
        self.ccost[a] += m.p.c0[v]
        for n in m.p.parents[v] + m.p.children[v]:
            if m.state[n] == EVICTED:
                a = self._merge(a, self.comp[self.node[n]])

    def neighbourhood_cost(self, x, m):
        seen = set()
        total = 0
        for n in m.p.parents[x] + m.p.children[x]:
            if m.state[n] == EVICTED:
                c = self.comp[self.node[n]]
                if c not in seen:
                    seen.add(c)
                    total += self.ccost[c]
        return total


def evicted_closure(prog, state, x):
    """e*(x): evicted ancestors through evicted parents, plus evicted
    descendants through evicted children (set semantics)."""
    seen = set()
    for nbrs in (prog.parents, prog.children):
        stack = [x]
        while stack:
            u = stack.pop()
            for v in nbrs[u]:
                if state[v] == EVICTED and v not in seen:
                    seen.add(v)
                    stack.append(v)
    return seen


def evicted_ancestors(prog, state, x):
    """e_R(x): the evicted tensors that rematerializing x would recompute
    (reachable from x through evicted parents)."""
    seen = set()
    stack = [x]
    while stack:
        u = stack.pop()
        for v in prog.parents[u]:
            if state[v] == EVICTED and v not in seen:
                seen.add(v)
                stack.append(v)
    return seen


def _mix64(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


IGNORE_SMALL, SAMPLE = 1, 2


def _searched(prog, m, cands, search, seed):
    """Candidates the search approximations leave (Appendix E): drop those
    below 1% of the pool's mean size; keep each with probability
    ceil(sqrt(n))/n by a SplitMix64 draw on its own stream; fall back to the
    non-small ones when nothing is left."""
    n = len(cands)
    total = sum(prog.size[x] for x in cands)
    big = [x for x in cands if not (search & IGNORE_SMALL) or 100 * prog.size[x] * n >= total]
    if not (search & SAMPLE):
        return big
    k = 0
    while k * k < n:
        k += 1
    if k >= n:
        return big
    tau = (k << 64) // n
    keep = [x for x in big
            if _mix64(((seed ^ 0xD6E8FEB86659FD93) + 0x9E3779B97F4A7C15 * ((m.evict_no << 32) + x)) & MASK64) < tau]
    return keep if keep else big


def visits(prog, m, x, heuristic):
    """The work counters of scoring candidate x: (members of the walked
    neighbourhood, neighbour slots examined).  e*(x) (h_DTR, h_{e*}, family
    cost e*) or e_R(x) (h_MSPS): its size and x's degree; union-find cost
    (h_DTR^eq, family cost eq): x's evicted parents and children, and its
    degree; other heuristics: none."""
    fc = (heuristic - 16) >> 2 if heuristic >= 16 else -1
    deg = len(prog.parents[x]) + len(prog.children[x])
    if heuristic in (0, 6) or fc == 0:
        return len(evicted_closure(prog, m.state, x)), deg
    if heuristic == 7:
        return len(evicted_ancestors(prog, m.state, x)), deg
    if heuristic == 1 or fc == 1:
        return sum(m.state[n] == EVICTED for n in prog.parents[x] + prog.children[x]), deg
    return 0, 0


def simulate(trace, budget: int, heuristic: int, seed: int = 0, policy: int = EAGER, search: int = 0) -> dict:
    """Heuristic-driven run of the same machine (h ids, policies and search
    flags as in the C-ABI)."""
    prog = Program(trace)
    fam = heuristic >= 16
    fc, fs, fm = ((heuristic - 16) >> 2, ((heuristic - 16) >> 1) & 1, (heuristic - 16) & 1) if fam else (-1, 0, 0)
    m = Machine(prog, budget, track_uf=(heuristic == 1 or fc == 1), policy=policy)
    c = None if m.oom else m.run()
    nbr = adj = 0
    while c is not None:
        best, bkey = None, None
        if search:
            c = _searched(prog, m, c, search, seed)
        for x in c:
            key = score_key(prog, m, x, heuristic, seed, m.clock - m.last[x])
            if bkey is None or key < bkey or (key == bkey and x < best):
                best, bkey = x, key
            v = visits(prog, m, x, heuristic)
            nbr += v[0]
            adj += v[1]
        m.n_scores += len(c)
        m.evict(best)
        c = m.run()
    status = 1 if m.oom else (2 if m.overflow else 0)
    # the operation being run when the simulation stopped: the bottom frame's
    # (the number of operations while the output condition runs)
    f0 = m.frames[0]
    failed = -1 if status == 0 else (f0[1] if f0[0] == "op" else prog.F)
    return dict(total_cost=m.cost, remat_cost=m.remat_cost, base_cost=m.cost - m.remat_cost,
                peak_memory=m.peak, final_memory=m.mem, n_executed_ops=m.n_exec,
                n_remats=m.n_remat, n_evictions=m.n_evict, n_eager_evictions=m.n_eager,
                n_scores=m.n_scores, n_nbr_visits=nbr, n_adj_visits=adj, status=status,
                failed_op=failed)


def score_key(prog, m, x, heuristic, seed, s):
    """Exact score of candidate x (a Fraction, or an int for h_rand) given its
    staleness s; prog supplies size, c0, parents and children, m the state,
    the union-find and the eviction number."""
    sz = prog.size[x]
    if heuristic in (0, 6):
        num = prog.c0[x] + sum(prog.c0[u] for u in evicted_closure(prog, m.state, x))
        return Fraction(num, sz * s) if heuristic == 0 else Fraction(num, sz)
    if heuristic == 1:
        return Fraction(prog.c0[x] + m.uf.neighbourhood_cost(x, m), sz * s)
    if heuristic == 2:
        return Fraction(prog.c0[x], sz * s)
    if heuristic == 3:
        return Fraction(1, s)
    if heuristic == 4:
        return Fraction(1, sz)
    if heuristic == 5:
        return _mix64((seed + 0x9E3779B97F4A7C15 * ((m.evict_no << 32) + x)) & MASK64)
    if heuristic == 7:
        return Fraction(prog.c0[x] + sum(prog.c0[u] for u in evicted_ancestors(prog, m.state, x)), sz)
    if heuristic < 16:
        raise ValueError(heuristic)
    fc, fs, fm = (heuristic - 16) >> 2, ((heuristic - 16) >> 1) & 1, (heuristic - 16) & 1
    if fc == 0:
        num = prog.c0[x] + sum(prog.c0[u] for u in evicted_closure(prog, m.state, x))
    elif fc == 1:
        num = prog.c0[x] + m.uf.neighbourhood_cost(x, m)
    elif fc == 2:
        num = prog.c0[x]
    else:
        num = 1
    return Fraction(num, (sz if fm else 1) * (s if fs else 1))
