"""Independent Python rendering of DTR over operator logs (Appendix C): the
log is lowered to storages, simulator tensors (a storage's root or a view of
it) and operators, and the eviction loop runs over storages.

  * lowering (Appendix C.6): CALL creates an operator whose outputs are new
    tensors, each a new storage (ALIAS to nothing) or a view of the viewed
    name's storage (size 0); MUTATE becomes a pure operator whose outputs are
    clones of the mutated inputs, and the mutated names are rebound to them;
    CONSTANT is a nullary operator of cost 0 whose storage is pinned; COPY,
    COPYFROM and RELEASE move external references; a storage whose external
    references drop to zero is released after the last operator issued.
    Tensors still referenced at the end must be defined and are locked.
  * storages (Appendix C.1): evictable = resident, unlocked, not pinned; a
    tensor is defined when its storage is resident and its operator ran after
    the storage last became resident.
  * rematerialization (Appendix C.4): lock the input storages, define the
    undefined inputs in listed order, allocate every non-view output, run,
    free the new copies of outputs that were already defined, unlock.
  * metadata (Appendix C.2, indexed by time): a tensor exists once its
    operator has first run; the cost of a storage sums, over its tensors that
    exist, the cost of each tensor's operator, and its dependencies are the
    storages those operators read; staleness uses the latest reference to any
    tensor of the storage.
  * banishing: a released storage is banished when no operation holds it and
    every tensor computed from it (outside the storage) is defined or gone;
    the resident storages of those tensors are then pinned.
"""
from __future__ import annotations

import copy

import brute
from brute import EVICTED, RESIDENT, UNCOMPUTED, BANISHED, EAGER, IGNORE, BANISH, CLOCK_LIMIT

MEMORY, ALIAS, CALL, MUTATE, CONSTANT, COPY, COPYFROM, RELEASE = range(8)


class StorageProgram:
    """The lowered log.  Per storage: size, c0 (cost of its root's operator),
    parents / children in the storage dependency graph, pinned (constant)."""

    def __init__(self, log):
        self.t_storage, self.t_op, self.t_alias = [], [], []
        self.size, self.const, self.root = [], [], []
        self.op_ins, self.op_outs, self.op_cost = [], [], []
        self.release = []                      # per op: storages released after it
        eref_t, eref_s = [], []
        names = {}

        def new_storage(size, const, root):
            self.size.append(size)
            self.const.append(const)
            self.root.append(root)
            eref_s.append(0)
            return len(self.size) - 1

        def new_tensor(storage, op, alias):
            self.t_storage.append(storage)
            self.t_op.append(op)
            self.t_alias.append(alias)
            eref_t.append(0)
            return len(self.t_storage) - 1

        def new_op(ins, cost):
            self.op_ins.append(list(ins))
            self.op_outs.append([])
            self.op_cost.append(cost)
            self.release.append([])
            return len(self.op_ins) - 1

        def inc(t):
            eref_t[t] += 1
            eref_s[self.t_storage[t]] += 1

        def dec(t):
            eref_t[t] -= 1
            s = self.t_storage[t]
            eref_s[s] -= 1
            assert eref_t[t] >= 0 and eref_s[s] >= 0
            if eref_s[s] == 0:
                self.release[-1].append(s)

        i, n = 0, log.n_instrs
        while i < n:
            k = int(log.kind[i])
            if k == CONSTANT:
                assert int(log.kind[i + 1]) == MEMORY and int(log.a[i + 1]) == int(log.a[i])
                o = new_op([], 0)
                t = new_tensor(-1, o, False)
                self.t_storage[t] = new_storage(int(log.value[i + 1]), True, t)
                self.op_outs[o].append(t)
                names[int(log.a[i])] = t
                inc(t)
                i += 2
            elif k == CALL:
                ins, outs = log.lists(i)
                o = new_op([names[int(x)] for x in ins], int(log.value[i]))
                local = {}
                for j, name in enumerate(outs):
                    mem, al = i + 1 + 2 * j, i + 2 + 2 * j
                    assert int(log.kind[mem]) == MEMORY and int(log.kind[al]) == ALIAS
                    src = int(log.b[al])
                    if src < 0:
                        t = new_tensor(-1, o, False)
                        self.t_storage[t] = new_storage(int(log.value[mem]), False, t)
                        local[int(name)] = t
                    else:
                        st = local[src] if src in local else names[src]
                        t = new_tensor(self.t_storage[st], o, True)
                    self.op_outs[o].append(t)
                for name, t in zip(outs, self.op_outs[o]):
                    names[int(name)] = t
                    inc(t)
                i += 1 + 2 * len(outs)
            elif k == MUTATE:
                ins, muts = log.lists(i)
                o = new_op([names[int(x)] for x in ins], int(log.value[i]))
                for m in muts:
                    old = names[int(m)]
                    t = new_tensor(-1, o, False)
                    self.t_storage[t] = new_storage(self.size[self.t_storage[old]], False, t)
                    self.op_outs[o].append(t)
                for m, t in zip(muts, self.op_outs[o]):
                    old = names[int(m)]
                    inc(t)
                    names[int(m)] = t
                    dec(old)
                i += 1
            elif k == COPY:
                t = names[int(log.b[i])]
                names[int(log.a[i])] = t
                inc(t)
                i += 1
            elif k == COPYFROM:
                old, t = names[int(log.a[i])], names[int(log.b[i])]
                inc(t)
                names[int(log.a[i])] = t
                dec(old)
                i += 1
            elif k == RELEASE:
                dec(names.pop(int(log.a[i])))
                i += 1
            else:
                raise ValueError(f"instruction {i}: unexpected kind {k}")
        self.required = [t for t in range(len(eref_t)) if eref_t[t] > 0]
        S = len(self.size)
        # tensors computed from each storage (outside it): what banishing must keep defined
        self.dep_tensors = [[] for _ in range(S)]
        for o in range(len(self.op_ins)):
            for u in self.op_ins[o]:
                p = self.t_storage[u]
                for v in self.op_outs[o]:
                    if self.t_storage[v] != p and v not in self.dep_tensors[p]:
                        self.dep_tensors[p].append(v)
        self.n = S


class LogMachine:
    def __init__(self, sp: StorageProgram, budget, heuristic, seed=0, policy=EAGER):
        # the storage graph that exists so far, grown as operators first run
        # (its cost c0, parents and children are what the scores read)
        self.p = copy.copy(sp)
        self.p.c0 = [0] * sp.n
        self.p.parents = [[] for _ in range(sp.n)]
        self.p.children = [[] for _ in range(sp.n)]
        self.budget, self.h, self.seed, self.policy = budget, heuristic, seed, policy
        S = sp.n
        self.state = [UNCOMPUTED] * S
        self.locks = [0] * S
        self.pinned = list(sp.const)
        self.pending = [False] * S
        self.sgen = [0] * S
        self.gen = [-1] * len(sp.t_storage)
        self.last = [0] * S
        self.mem = self.peak = self.clock = self.cost = self.remat_cost = 0
        self.n_exec = self.n_remat = self.n_evict = self.n_eager = self.n_scores = 0
        self.evict_no = 0
        self.stop = None                     # "oom" or "clock"
        fc = (heuristic - 16) >> 2 if heuristic >= 16 else -1
        self.uf = brute.UnionFind() if (heuristic == 1 or fc == 1) else None
        self.cur = 0

    def defined(self, t):
        s = self.p.t_storage[t]
        return self.state[s] == RESIDENT and self.gen[t] == self.sgen[s]

    def evictable(self, s):
        return self.state[s] == RESIDENT and self.locks[s] == 0 and not self.pinned[s]

    def evict(self, s, eager):
        self.state[s] = EVICTED
        self.mem -= self.p.size[s]
        if eager:
            self.n_eager += 1
        else:
            self.n_evict += 1
            self.evict_no += 1
        if self.uf is not None:
            self.uf.on_evict(s, self)

    def allocate(self, need):
        while self.mem + need > self.budget:
            cands = [s for s in range(self.p.n) if self.evictable(s)]
            if not cands:
                self.stop = "oom"
                return False
            best, bkey = None, None
            for s in cands:
                key = brute.score_key(self.p, self, s, self.h, self.seed, self.clock - self.last[s])
                if bkey is None or key < bkey or (key == bkey and s < best):
                    best, bkey = s, key
            self.n_scores += len(cands)
            self.evict(best, False)
        return True

    def banish(self, s):
        p = self.p
        if self.locks[s] > 0 or not all(self.defined(v) or self.state[p.t_storage[v]] == BANISHED
                                        for v in p.dep_tensors[s]):
            self.pending[s] = True
            return
        self.pending[s] = False
        if self.state[s] == RESIDENT:
            self.mem -= p.size[s]
        self.state[s] = BANISHED
        self.n_eager += 1
        for v in p.dep_tensors[s]:
            if self.state[p.t_storage[v]] == RESIDENT:
                self.pinned[p.t_storage[v]] = True

    def call(self, o, remat):
        p = self.p
        ins = p.op_ins[o]
        for u in ins:
            assert self.state[p.t_storage[u]] != BANISHED
            self.locks[p.t_storage[u]] += 1
        for u in ins:
            if not self.defined(u):
                if not self.call(p.t_op[u], True):
                    return False
        roots = [v for v in p.op_outs[o] if not p.t_alias[v]]
        need = sum(p.size[p.t_storage[v]] for v in roots)
        if not self.allocate(need):
            return False
        for u in ins:
            self.last[p.t_storage[u]] = self.clock
        for v in p.op_outs[o]:
            self.last[p.t_storage[v]] = self.clock
        c = p.op_cost[o]
        self.clock += c
        self.cost += c
        self.n_exec += 1
        if remat:
            self.remat_cost += c
            self.n_remat += 1
        self.mem += need
        self.peak = max(self.peak, self.mem)
        for v in roots:
            s = p.t_storage[v]
            if self.state[s] == RESIDENT:
                self.mem -= p.size[s]                     # the new copy of a defined output
            else:
                was_evicted = self.state[s] == EVICTED
                self.state[s] = RESIDENT
                self.sgen[s] += 1
                self.gen[v] = self.sgen[s]
                if self.uf is not None:
                    self.uf.on_materialize(s, was_evicted, self)
        for v in p.op_outs[o]:
            if p.t_alias[v]:
                self.gen[v] = self.sgen[p.t_storage[v]]
        if not remat:
            # the operator's tensors exist from now on
            for v in p.op_outs[o]:
                s = p.t_storage[v]
                if not p.const[s]:
                    p.c0[s] += c
                for u in ins:
                    q = p.t_storage[u]
                    if q != s and q not in p.parents[s]:
                        p.parents[s].append(q)
                        p.children[q].append(s)
        if self.clock >= CLOCK_LIMIT:
            self.stop = "clock"
            return False
        for u in ins:
            self.locks[p.t_storage[u]] -= 1
        if remat and self.policy == BANISH:
            for u in ins:
                if self.pending[p.t_storage[u]]:
                    self.banish(p.t_storage[u])
        return True

    def run(self):
        p = self.p
        for o in range(len(p.op_ins)):
            self.cur = o
            if not self.call(o, False):
                return
            for s in p.release[o]:
                if self.policy == EAGER:
                    if self.evictable(s):
                        self.evict(s, True)
                elif self.policy == BANISH:
                    self.banish(s)
        self.cur = len(p.op_ins)
        for t in p.required:
            self.locks[p.t_storage[t]] += 1
            if not self.defined(t) and not self.call(p.t_op[t], True):
                return


def simulate(log, budget, heuristic, seed=0, policy=EAGER) -> dict:
    sp = StorageProgram(log)
    m = LogMachine(sp, budget, heuristic, seed, policy)
    m.run()
    status = {None: 0, "oom": 1, "clock": 2}[m.stop]
    return dict(total_cost=m.cost, remat_cost=m.remat_cost, base_cost=m.cost - m.remat_cost,
                peak_memory=m.peak, final_memory=m.mem, n_executed_ops=m.n_exec, n_remats=m.n_remat,
                n_evictions=m.n_evict, n_eager_evictions=m.n_eager, n_scores=m.n_scores, status=status,
                failed_op=-1 if m.stop is None else m.cur)
