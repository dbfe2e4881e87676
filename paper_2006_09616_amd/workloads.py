"""Seeded synthetic operator traces and simulation batches for the DTR eviction loop.

This module only builds *programs*: operators with input tensor ids, integer
output sizes and integer compute costs, plus flags (constant, required output).
It holds no part of the eviction method itself.  The one derived quantity it
computes is a program's natural peak memory when every tensor is freed right
after its last use (reference counting, no eviction), because the workloads
space their memory budgets as fractions of that peak.

Both the HIP path and the CPU oracle consume exactly these arrays, so the
floating-point draws used for sizes (log-normal) cannot break parity: they are
taken once, here, and rounded to integers.

Trace model (single output per operator, as the method assumes in Section 2):
  * tensors 0..n_tensors-1; operators 0..n_ops-1 in execution order;
  * op o produces tensor ``op_output[o]`` from ``op_inputs[off[o]:off[o+1]]``;
  * a tensor flagged CONSTANT has no producer and is resident from time 0;
  * a tensor flagged REQUIRED_OUTPUT is never released and must be resident
    when the program ends.

The backward pass follows the gradient program of Appendix A (network
definition): for each forward operator f_j, visited in reverse, the gradient
operator reads f_j's inputs and the gradients of every operator that consumed
f_j's output, and produces a gradient of the same size as that output.
"""
from __future__ import annotations

import hashlib
import math
from dataclasses import dataclass, field

import numpy as np

FLAG_CONSTANT = 1
FLAG_REQUIRED = 2

# heuristic ids (shared numbering with the C-ABI; the numbers carry no arithmetic)
H_DTR, H_EQ, H_LOCAL, H_LRU, H_SIZE, H_RAND, H_ESTAR, H_MSPS = range(8)
HEURISTIC_NAMES = ["dtr", "eq", "local", "lru", "size", "rand", "estar", "msps"]
# the ablation family h'(s, m, c): cost measure c, staleness s and size m each
# used (1) or ablated (0); id = H_FAMILY + 4*c + 2*s + m
C_ESTAR, C_EQCLASS, C_LOCAL, C_NONE = range(4)
H_FAMILY = 16


def h_family(c: int, s: int, m: int) -> int:
    assert 0 <= c < 4 and s in (0, 1) and m in (0, 1)
    return H_FAMILY + 4 * c + 2 * s + m


ALL_FAMILY = [h_family(c, s, m) for c in range(4) for s in (0, 1) for m in (0, 1)]

BUDGET_UNLIMITED = (1 << 63) - 1

# deallocation policies (what a release does): evict eagerly, nothing, banish
POLICY_EAGER, POLICY_IGNORE, POLICY_BANISH = range(3)
# search approximation flags: ignore small candidates, search a random sample
SEARCH_IGNORE_SMALL, SEARCH_SAMPLE = 1, 2

SPEC_DTYPE = np.dtype([("trace", "<i4"), ("heuristic", "<i4"),
                       ("budget", "<i8"), ("seed", "<u8"),
                       ("policy", "<i4"), ("search", "<i4")])


def make_specs(rows) -> np.ndarray:
    """Simulation specs from rows (trace, heuristic, budget, seed[, policy[, search]])."""
    a = np.zeros(len(rows), dtype=SPEC_DTYPE)
    for i, r in enumerate(rows):
        a[i] = (r[0], r[1], r[2], r[3], r[4] if len(r) > 4 else POLICY_EAGER, r[5] if len(r) > 5 else 0)
    return a


@dataclass
class Trace:
    name: str
    tensor_size: np.ndarray        # int64 [n_tensors]
    tensor_flags: np.ndarray       # uint8 [n_tensors]
    op_output: np.ndarray          # int32 [n_ops]
    op_cost: np.ndarray            # int64 [n_ops]
    op_input_offsets: np.ndarray   # int64 [n_ops + 1]
    op_inputs: np.ndarray          # int32 [n_edges]
    meta: dict = field(default_factory=dict)

    def __post_init__(self):
        self.tensor_size = np.ascontiguousarray(self.tensor_size, dtype=np.int64)
        self.tensor_flags = np.ascontiguousarray(self.tensor_flags, dtype=np.uint8)
        self.op_output = np.ascontiguousarray(self.op_output, dtype=np.int32)
        self.op_cost = np.ascontiguousarray(self.op_cost, dtype=np.int64)
        self.op_input_offsets = np.ascontiguousarray(self.op_input_offsets, dtype=np.int64)
        self.op_inputs = np.ascontiguousarray(self.op_inputs, dtype=np.int32)

    @property
    def n_tensors(self) -> int:
        return int(self.tensor_size.shape[0])

    @property
    def n_ops(self) -> int:
        return int(self.op_output.shape[0])

    def inputs(self, o: int) -> np.ndarray:
        return self.op_inputs[self.op_input_offsets[o]:self.op_input_offsets[o + 1]]

    def digest(self) -> str:
        h = hashlib.sha256()
        for a in (self.tensor_size, self.tensor_flags, self.op_output, self.op_cost,
                  self.op_input_offsets, self.op_inputs):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


@dataclass
class Workload:
    name: str
    traces: list
    specs: np.ndarray              # SPEC_DTYPE [n_sims]
    peaks: list                    # natural peak per trace
    description: str = ""

    @property
    def n_sims(self) -> int:
        return int(self.specs.shape[0])

    def digest(self) -> str:
        h = hashlib.sha256()
        for t in self.traces:
            h.update(t.digest().encode())
        h.update(self.specs.tobytes())
        return h.hexdigest()


# ----------------------------------------------------------------------------
# program construction helpers
# ----------------------------------------------------------------------------

def _csr(lists):
    lens = np.fromiter((len(x) for x in lists), dtype=np.int64, count=len(lists))
    off = np.zeros(len(lists) + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    flat = np.fromiter((v for x in lists for v in x), dtype=np.int32, count=int(off[-1]))
    return off, flat


def _segment_gather(starts, lens):
    """Indices of the concatenation of ranges [starts[i], starts[i]+lens[i])."""
    lens = np.asarray(lens, dtype=np.int64)
    total = int(lens.sum())
    if total == 0:
        return np.zeros(0, dtype=np.int64)
    seg_off = np.zeros(len(lens), dtype=np.int64)
    np.cumsum(lens[:-1], out=seg_off[1:])
    return np.repeat(np.asarray(starts, dtype=np.int64) - seg_off, lens) + np.arange(total, dtype=np.int64)


def with_backward(fwd_off, fwd_in, fwd_size, fwd_cost, bwd_cost, name="", meta=None):
    """Forward program (tensor id == op index) followed by its gradient program.

    Gradient operator for f_j (emitted for j = F-1 down to 0) reads
    inputs(f_j) in their listed order, then the gradients of f_j's consumers
    in ascending consumer order; it outputs a tensor of size(y_j).  Gradients
    of nullary forward operators are the program's required outputs.
    """
    fwd_off = np.asarray(fwd_off, dtype=np.int64)
    fwd_in = np.asarray(fwd_in, dtype=np.int64)
    F = len(fwd_off) - 1
    n_in = np.diff(fwd_off)
    reader = np.repeat(np.arange(F, dtype=np.int64), n_in)          # consumer op of each edge
    order = np.lexsort((reader, fwd_in))                            # by producer j, then consumer c
    cons_c = reader[order]
    n_cons = np.bincount(fwd_in, minlength=F).astype(np.int64)
    cons_off = np.zeros(F + 1, dtype=np.int64)
    np.cumsum(n_cons, out=cons_off[1:])

    js = np.arange(F - 1, -1, -1, dtype=np.int64)                   # backward op b handles j = F-1-b
    len1 = n_in[js]
    len2 = n_cons[js]
    blen = len1 + len2
    boff = np.zeros(F + 1, dtype=np.int64)
    np.cumsum(blen, out=boff[1:])
    bin_ = np.empty(int(boff[-1]), dtype=np.int64)
    pos1 = _segment_gather(boff[:-1], len1)
    bin_[pos1] = fwd_in[_segment_gather(fwd_off[js], len1)]
    pos2 = _segment_gather(boff[:-1] + len1, len2)
    bin_[pos2] = F + (F - 1 - cons_c[_segment_gather(cons_off[js], len2)])

    n = 2 * F
    size = np.empty(n, dtype=np.int64)
    size[:F] = fwd_size
    size[F:] = np.asarray(fwd_size, dtype=np.int64)[js]
    cost = np.empty(n, dtype=np.int64)
    cost[:F] = fwd_cost
    cost[F:] = bwd_cost
    flags = np.zeros(n, dtype=np.uint8)
    nullary = np.nonzero(n_in == 0)[0]
    flags[F + (F - 1 - nullary)] |= FLAG_REQUIRED
    off = np.concatenate([fwd_off, fwd_off[-1] + boff[1:]])
    inp = np.concatenate([fwd_in, bin_]).astype(np.int32)
    return Trace(name, size, flags, np.arange(n, dtype=np.int32), cost, off, inp,
                 meta=dict(meta or {}, n_forward=F))


def natural_peak(tr: Trace) -> int:
    """Peak memory of the program when each tensor is freed right after its
    last reader (or right after it is produced, if nothing reads it); constants
    and required outputs are never freed.  No eviction is involved: this is the
    program's own memory profile, used to space budgets."""
    n, F = tr.n_tensors, tr.n_ops
    last = np.full(n, -1, dtype=np.int64)
    prod = np.full(n, -1, dtype=np.int64)
    prod[tr.op_output] = np.arange(F)
    reader = np.repeat(np.arange(F, dtype=np.int64), np.diff(tr.op_input_offsets))
    np.maximum.at(last, tr.op_inputs.astype(np.int64), reader)
    last = np.maximum(last, prod)
    const = (tr.tensor_flags & FLAG_CONSTANT) != 0
    keep = const | ((tr.tensor_flags & FLAG_REQUIRED) != 0)
    freed = ~keep & (last >= 0)
    free_at = np.zeros(F, dtype=np.int64)
    np.add.at(free_at, last[freed], tr.tensor_size[freed])
    alloc = tr.tensor_size[tr.op_output]
    base = int(tr.tensor_size[const].sum())
    before_free = base + np.cumsum(alloc) - np.concatenate([[0], np.cumsum(free_at)[:-1]])
    return int(max(base, int(before_free.max()) if F else base))


def linear_budgets(peak: int, lo_pct: int, hi_pct: int, k_count: int):
    """k_count budgets linearly spaced from lo_pct% to hi_pct% of peak, each
    rounded down, in exact integer arithmetic."""
    if k_count == 1:
        return [peak * hi_pct // 100]
    den = 100 * (k_count - 1)
    return [peak * (lo_pct * (k_count - 1) + (hi_pct - lo_pct) * k) // den for k in range(k_count)]


def splitmix64(x: int) -> int:
    """SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014): one
    increment by the golden-ratio gamma, then the variant-13 finaliser.  Used
    here only to derive per-tree seeds."""
    m = (1 << 64) - 1
    z = (x + 0x9E3779B97F4A7C15) & m
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return z ^ (z >> 31)


def _specs(rows):
    return make_specs(rows)


# ----------------------------------------------------------------------------
# workload 1: linear feed-forward chain (Appendix A network)
# ----------------------------------------------------------------------------

def chain_trace(N: int, size: int = 1, cost: int = 1) -> Trace:
    """f_1 nullary, f_i(t_{i-1}); gradient ops as in Appendix A.  Tensor ids:
    t_i -> i-1, gradient of f_i -> N + (N - i)."""
    off = np.arange(N + 1, dtype=np.int64) - 1
    off[0] = 0
    inp = np.arange(N - 1, dtype=np.int64)        # f_{i+1} reads t_i  (id i-1)
    return with_backward(off, inp, np.full(N, size, np.int64), np.full(N, cost, np.int64),
                         np.full(N, cost, np.int64), name=f"chain{N}", meta=dict(N=N))


def shared_weight_chain(N: int, weight_size: int = 1, constant: bool = True) -> Trace:
    """The Appendix A chain in which every forward and gradient operator also
    reads one weight W (one weight shared by every layer, as in the recurrent
    and tree-structured models of Section 4).  Tensor ids as in chain_trace,
    W is id 2N: a constant, or (constant=False) the output of a nullary
    operator of cost 1 run first, so that W is evictable whenever no operator
    holds it."""
    tr = chain_trace(N)
    n = tr.n_tensors
    lists = [list(tr.inputs(o)) + [n] for o in range(tr.n_ops)]
    outs, costs = tr.op_output.copy(), tr.op_cost.copy()
    if not constant:
        lists = [[]] + lists
        outs = np.concatenate([[n], outs]).astype(np.int32)
        costs = np.concatenate([[1], costs]).astype(np.int64)
    off, flat = _csr(lists)
    size = np.concatenate([tr.tensor_size, [weight_size]]).astype(np.int64)
    flags = np.concatenate([tr.tensor_flags, [FLAG_CONSTANT if constant else 0]]).astype(np.uint8)
    return Trace(f"chainW{N}" + ("" if constant else "op"), size, flags, outs, costs, off, flat,
                 meta=dict(N=N, weight=n))


def plain_chain(n_ops: int, cost: int, last_reads_first: bool = False, required=(-1,)) -> Trace:
    """Forward-only chain t_0 = f_0(), t_i = f_i(t_{i-1}), unit sizes, every
    operator of the given cost; with last_reads_first the last operator reads
    (t_0, t_{n-2}).  `required` lists the tensor ids (negative: from the end)
    that are required outputs."""
    ins = [[]] + [[i - 1] for i in range(1, n_ops)]
    if last_reads_first and n_ops >= 3:
        ins[-1] = [0, n_ops - 2]
    off, flat = _csr(ins)
    flags = np.zeros(n_ops, np.uint8)
    for t in required:
        flags[t % n_ops] |= FLAG_REQUIRED
    return Trace(f"plainchain{n_ops}", np.ones(n_ops, np.int64), flags, np.arange(n_ops, dtype=np.int32),
                 np.full(n_ops, cost, np.int64), off, flat)


def near_tie_program(seed: int, k: int = 24, fillers: int = 2048) -> Trace:
    """Eviction decisions between large, nearly equal scores.  k tensors x_i
    (sizes near 2^35 or 2^34, some equal, some exactly double another's with
    double the cost; costs from 1 to 2^28, some equal) are made first, some
    pairs are read together by one operator (equal last access), x's of equal
    cost per byte are read one after another by cheap operators, then a chain
    of `fillers` operators of cost 2^28 and size 1 moves the clock to about
    2^39, so staleness values differ by 1 to 2^28 in about 2^39.  Nullary
    operators G then need a third of the x memory (pieces below 2^36), and
    every x is read again (in a shuffled order) while the G outputs are still
    held, so the x's are evicted and rematerialized by decisions among
    near-ties.  The budget of the workload is
    the sum of the x sizes plus 4 (see near_tie_budgets)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    big = 1 << 35
    sizes, costs, lists = [], [], []
    for i in range(k):
        r = rng.integers(0, 4)
        if r == 0 and i >= 2:            # (2c, 2m) against an earlier (c, m): an exact tie of c/m
            j = int(rng.integers(0, i))
            if sizes[j] < big and 2 * costs[j] <= (1 << 28):
                sizes.append(2 * sizes[j])
                costs.append(2 * costs[j])
            else:
                sizes.append(sizes[j])
                costs.append(costs[j])
        elif r == 1 and i >= 1:          # a copy of an earlier (c, m)
            j = int(rng.integers(0, i))
            sizes.append(sizes[j])
            costs.append(costs[j])
        else:
            base = big if rng.integers(0, 2) else big // 2
            sizes.append(base - int(rng.integers(0, 1 << int(rng.integers(0, 31)))))
            costs.append(int(rng.integers(1, (1 << 28) + 1)) if rng.integers(0, 2)
                         else (1 << 19) * int(rng.integers(1, 9)) + int(rng.integers(0, 4)))
        n_in = int(rng.integers(0, min(2, i) + 1))
        lists.append(sorted(int(v) for v in rng.choice(i, size=n_in, replace=False)) if n_in else [])
    out_size = list(sizes)
    out_cost = list(costs)
    # pairs read together (equal last access); outputs of size 1 released at once
    for _ in range(k // 4):
        a, b = sorted(int(v) for v in rng.choice(k, size=2, replace=False))
        lists.append([a, b])
        out_size.append(1)
        out_cost.append(int(rng.integers(1, 1 << 20)))
    # x's of equal (c, m) or (2c, 2m) read one after another by cheap
    # operators: their staleness values end up a few units apart
    same = [(a, b) for b in range(k) for a in range(b) if sizes[a] * costs[b] == sizes[b] * costs[a]]
    for a, b in same[:6]:
        for x in (a, b):
            lists.append([x])
            out_size.append(1)
            out_cost.append(int(rng.integers(1, 65)))
    # the filler chain
    h0 = len(lists)
    for j in range(fillers):
        lists.append([] if j == 0 else [h0 + j - 1])
        out_size.append(1)
        out_cost.append(1 << 28)
    # G: a third of the x memory, in pieces below the size limit of 2^36,
    # made by nullary operators (so that rematerializing them is cheap)
    g = len(lists)
    need = int(sum(sizes)) // 3
    n_g = -(-need // ((1 << 36) - 1))
    for _ in range(n_g):
        lists.append([])
        out_size.append(need // n_g)
        out_cost.append(int(rng.integers(1, 1 << 20)))
    z = len(lists)
    for i in rng.permutation(k):
        lists.append([int(i)])
        out_size.append(1)
        out_cost.append(int(rng.integers(1, 1 << 20)))
    lists.append(list(range(g, g + n_g)))
    out_size.append(1)
    out_cost.append(1)
    n = len(lists)
    flags = np.zeros(n, np.uint8)
    flags[z:] = FLAG_REQUIRED
    off, flat = _csr(lists)
    return Trace(f"neartie{seed}", np.asarray(out_size, np.int64), flags, np.arange(n, dtype=np.int32),
                 np.asarray(out_cost, np.int64), off, flat, meta=dict(seed=seed, k=k))


def near_tie_budgets(tr: Trace) -> list:
    """Budgets of a near_tie_program: the x memory plus 4 units, and that
    less 1/16 and 1/8 of the largest x (more evictions per decision)."""
    k = tr.meta["k"]
    xs = tr.tensor_size[:k]
    b = int(xs.sum()) + 4
    return [b, b - int(xs.max()) // 16, b - int(xs.max()) // 8]


def config_chain(N: int = 32) -> Workload:
    tr = chain_trace(N)
    peak = natural_peak(tr)
    budgets = [math.ceil(2 * math.sqrt(N)), 16, 32, 64, BUDGET_UNLIMITED]
    specs = _specs([(0, H_DTR, b, (1 << 32) + i) for i, b in enumerate(budgets)])
    return Workload("chain32", [tr], specs, [peak],
                    f"linear chain N={N}, unit sizes/costs, h_DTR at 5 budgets")


# ----------------------------------------------------------------------------
# workload 2: ResNet-like residual stack
# ----------------------------------------------------------------------------

MiB = 1 << 20


def resnet_trace(seed: int = 2, blocks: int = 50) -> Trace:
    rng = np.random.Generator(np.random.PCG64(seed))
    ins = [[]]                                    # op 0: network input (nullary)
    for b in range(blocks):
        x = len(ins) - 1
        base = len(ins)
        ins.append([x])                           # conv1
        ins.append([base])                        # bn1
        ins.append([base + 1])                    # relu
        ins.append([base + 2])                    # conv2
        ins.append([base + 3])                    # bn2
        ins.append([base + 4, x])                 # add(bn2, block input)
    ins.append([len(ins) - 1])                    # loss
    F = len(ins)
    off, flat = _csr(ins)
    size = np.maximum(1, np.rint(rng.lognormal(math.log(4 * MiB), 1.0, size=F - 1))).astype(np.int64)
    size = np.concatenate([size, [4]])
    fcost = np.maximum(1, size // 4096) * rng.integers(1, 5, size=F)
    fcost[-1] = 1
    bsize = size[::-1]
    bcost = np.maximum(1, bsize // 4096) * rng.integers(1, 5, size=F)
    return with_backward(off, flat, size, fcost, bcost, name=f"resnet{blocks}",
                         meta=dict(seed=seed, blocks=blocks))


def config_resnet() -> Workload:
    tr = resnet_trace()
    peak = natural_peak(tr)
    budgets = linear_budgets(peak, 10, 100, 256)
    rows = []
    for h in (H_DTR, H_EQ, H_LOCAL, H_LRU, H_SIZE, H_RAND):
        for b in budgets:
            rows.append((0, h, b, 2 * (1 << 32) + len(rows)))
    return Workload("resnet50blk", [tr], _specs(rows), [peak],
                    "ResNet-like 50 residual blocks, 256 budgets x 6 heuristics")


# ----------------------------------------------------------------------------
# workload 3: transformer encoder
# ----------------------------------------------------------------------------

def transformer_trace(layers=12, hidden=768, seq=512, batch=8, heads=12, elem=2) -> Trace:
    B, S, H = batch, seq, hidden
    d = H // heads
    M = B * S

    def cst(flops):
        return max(1, int(round(flops / 1e6)))

    ins, size, cost = [], [], []

    def op(inputs, nbytes, c):
        ins.append(list(inputs))
        size.append(int(nbytes))
        cost.append(int(c))
        return len(ins) - 1

    x = op([], M * H * elem, cst(M * H))                                  # embedding
    for _ in range(layers):
        ln1 = op([x], M * H * elem, cst(8 * M * H))
        qkv = op([ln1], M * 3 * H * elem, cst(2 * M * H * 3 * H))
        ctxs = []
        for _h in range(heads):
            sc = op([qkv], B * S * S * elem, cst(2 * B * S * S * d))
            sm = op([sc], B * S * S * elem, cst(5 * B * S * S))
            ctxs.append(op([sm, qkv], M * d * elem, cst(2 * B * S * S * d)))
        cat = op(ctxs, M * H * elem, cst(M * H))
        proj = op([cat], M * H * elem, cst(2 * M * H * H))
        add1 = op([proj, x], M * H * elem, cst(M * H))
        ln2 = op([add1], M * H * elem, cst(8 * M * H))
        mlp1 = op([ln2], M * 4 * H * elem, cst(2 * M * H * 4 * H))
        gelu = op([mlp1], M * 4 * H * elem, cst(8 * M * 4 * H))
        mlp2 = op([gelu], M * H * elem, cst(2 * M * 4 * H * H))
        x = op([mlp2, add1], M * H * elem, cst(M * H))
    op([x], 4, cst(M * H))                                               # loss
    off, flat = _csr(ins)
    fcost = np.asarray(cost, dtype=np.int64)
    return with_backward(off, flat, np.asarray(size, np.int64), fcost, 2 * fcost[::-1],
                         name=f"transformer{layers}",
                         meta=dict(layers=layers, hidden=H, seq=S, batch=B, heads=heads))


def config_transformer() -> Workload:
    tr = transformer_trace()
    peak = natural_peak(tr)
    budgets = linear_budgets(peak, 15, 100, 512)
    rows = []
    for h in (H_DTR, H_EQ, H_LRU):
        for b in budgets:
            rows.append((0, h, b, 3 * (1 << 32) + len(rows)))
    return Workload("transformer12", [tr], _specs(rows), [peak],
                    "transformer encoder 12 layers, 512 budgets x 3 heuristics")


# ----------------------------------------------------------------------------
# workload 4: TreeLSTM over random binary trees
# ----------------------------------------------------------------------------

def treelstm_trace(seed: int, hidden: int = 256, min_leaves=64, max_leaves=512) -> Trace:
    rng = np.random.Generator(np.random.PCG64(seed))
    L = int(rng.integers(min_leaves, max_leaves + 1))
    H = hidden
    g_bytes, h_bytes = 5 * H * 4, H * 4
    ins, size, cost = [], [], []

    def op(inputs, nbytes, c):
        ins.append(inputs)
        size.append(nbytes)
        cost.append(c)
        return len(ins) - 1

    def cst(flops):
        return max(1, int(round(flops / 1e3)))

    # shape: pre-order split draws, post-order emission
    def build(n_leaves):
        if n_leaves == 1:
            g = op([], g_bytes, cst(2 * 5 * H * H))
            a = op([g], g_bytes, cst(4 * 5 * H))
            c = op([a], h_bytes, cst(5 * H))
            tc = op([c], h_bytes, cst(H))
            h = op([a, tc], h_bytes, cst(H))
            return h, c
        k = int(rng.integers(1, n_leaves))
        hl, cl = build(k)
        hr, cr = build(n_leaves - k)
        g = op([hl, hr], g_bytes, cst(2 * 5 * H * 2 * H))
        a = op([g], g_bytes, cst(4 * 5 * H))
        c = op([a, cl, cr], h_bytes, cst(5 * H))
        tc = op([c], h_bytes, cst(H))
        h = op([a, tc], h_bytes, cst(H))
        return h, c

    hroot, _ = build(L)
    op([hroot], 4, 1)                                                    # loss
    off, flat = _csr(ins)
    fcost = np.asarray(cost, dtype=np.int64)
    return with_backward(off, flat, np.asarray(size, np.int64), fcost, 2 * fcost[::-1],
                         name=f"treelstm_L{L}", meta=dict(seed=seed, leaves=L, hidden=H))


def config_treelstm(n_trees: int = 4096, budgets_per_tree: int = 8) -> Workload:
    import sys
    old = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old, 5000))
    try:
        traces = [treelstm_trace(splitmix64(4 * (1 << 32) + i)) for i in range(n_trees)]
    finally:
        sys.setrecursionlimit(old)
    peaks = [natural_peak(t) for t in traces]
    rows = []
    for i, p in enumerate(peaks):
        for b in linear_budgets(p, 20, 100, budgets_per_tree):
            rows.append((i, H_EQ, b, 4 * (1 << 32) + len(rows)))
    return Workload(f"treelstm{n_trees}", traces, _specs(rows), peaks,
                    f"{n_trees} TreeLSTM traces x {budgets_per_tree} budgets, h_DTR^eq")


# ----------------------------------------------------------------------------
# workload 5: large random DAG with a locality window
# ----------------------------------------------------------------------------

def random_dag_trace(seed: int = 5, n_forward: int = 100_000, window: int = 64,
                     max_in: int = 3, median_bytes: int = MiB, sigma: float = 1.5,
                     cost_mult: int = 8) -> Trace:
    rng = np.random.Generator(np.random.PCG64(seed))
    ins = [[]]
    for k in range(1, n_forward):
        lo = max(0, k - window)
        w = k - lo
        n = min(int(rng.integers(1, max_in + 1)), k)
        pick = rng.choice(w, size=n, replace=False) + lo
        ins.append(sorted(int(v) for v in pick))
    off, flat = _csr(ins)
    size = np.maximum(1, np.rint(rng.lognormal(math.log(median_bytes), sigma, size=n_forward))).astype(np.int64)
    fcost = np.maximum(1, size // 4096) * rng.integers(1, cost_mult + 1, size=n_forward)
    bsize = size[::-1]
    bcost = np.maximum(1, bsize // 4096) * rng.integers(1, cost_mult + 1, size=n_forward)
    return with_backward(off, flat, size, fcost, bcost, name=f"randdag{n_forward}",
                         meta=dict(seed=seed, n_forward=n_forward, window=window))


def config_random_dag(n_forward: int = 100_000, n_budgets: int = 1024, lo_pct: int = 5) -> Workload:
    tr = random_dag_trace(n_forward=n_forward)
    peak = natural_peak(tr)
    rows = [(0, H_DTR, b, 5 * (1 << 32) + i)
            for i, b in enumerate(linear_budgets(peak, lo_pct, 100, n_budgets))]
    return Workload(f"randdag{n_forward}", [tr], _specs(rows), [peak],
                    f"random DAG {n_forward} fwd ops, {n_budgets} budgets, h_DTR")


# ----------------------------------------------------------------------------
# small random programs for differential tests
# ----------------------------------------------------------------------------

def random_program(seed: int, n_ops: int, n_const: int = 0, max_in: int = 3,
                   max_size: int = 8, max_cost: int = 5, p_required: float = 0.1,
                   backward: bool = False, window: int | None = None,
                   permute_ids: bool = True) -> Trace:
    """Random DAG program.  Constants and operator outputs are interleaved in
    execution order, then tensor ids are optionally shuffled, so id order and
    execution order differ (this exercises the id tie-break and id mapping)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if backward:
        ins = [[]]
        for k in range(1, n_ops):
            lo = 0 if window is None else max(0, k - window)
            w = k - lo
            n = int(rng.integers(0, min(max_in, w) + 1))
            pick = rng.choice(w, size=n, replace=False) + lo if n else []
            ins.append(sorted(int(v) for v in pick))
        off, flat = _csr(ins)
        size = rng.integers(1, max_size + 1, size=n_ops)
        fcost = rng.integers(1, max_cost + 1, size=n_ops)
        bcost = rng.integers(1, max_cost + 1, size=n_ops)
        tr = with_backward(off, flat, size, fcost, bcost, name=f"rand_bwd{seed}")
        sizes, flags = tr.tensor_size.copy(), tr.tensor_flags.copy()
        outs, costs = tr.op_output.copy(), tr.op_cost.copy()
        off2, inp2 = tr.op_input_offsets.copy(), tr.op_inputs.copy()
    else:
        # execution order over "slots": each slot is a constant or an operator output
        kinds = np.array([1] * n_const + [0] * n_ops)
        rng.shuffle(kinds)
        sizes = rng.integers(1, max_size + 1, size=len(kinds)).astype(np.int64)
        flags = np.where(kinds == 1, FLAG_CONSTANT, 0).astype(np.uint8)
        outs, costs, lists = [], [], []
        for slot, k in enumerate(kinds):
            if k == 1:
                continue
            lo = 0 if window is None else max(0, slot - window)
            avail = np.arange(lo, slot)
            n = int(rng.integers(0, min(max_in, len(avail)) + 1))
            pick = sorted(int(v) for v in rng.choice(avail, size=n, replace=False)) if n else []
            lists.append(pick)
            outs.append(slot)
            costs.append(int(rng.integers(1, max_cost + 1)))
        req = rng.random(len(kinds)) < p_required
        flags[(kinds == 0) & req] |= FLAG_REQUIRED
        off2, inp2 = _csr(lists)
        outs = np.asarray(outs, np.int32)
        costs = np.asarray(costs, np.int64)
    if permute_ids:
        n = len(sizes)
        perm = rng.permutation(n)            # old id -> new id
        new_sizes = np.empty_like(sizes)
        new_flags = np.empty_like(flags)
        new_sizes[perm] = sizes
        new_flags[perm] = flags
        sizes, flags = new_sizes, new_flags
        outs = perm[np.asarray(outs)]
        inp2 = perm[np.asarray(inp2)] if len(inp2) else np.asarray(inp2)
        # the gradient op may list inputs in any order; keep listed order
    return Trace(f"rand{seed}", sizes, flags, outs, costs, off2, inp2, meta=dict(seed=seed))


CONFIGS = {
    "chain32": config_chain,
    "resnet50blk": config_resnet,
    "transformer12": config_transformer,
    "treelstm4096": config_treelstm,
    "randdag100k": config_random_dag,
}


def make_config(name: str, **kw) -> Workload:
    return CONFIGS[name](**kw)


# ----------------------------------------------------------------------------
# operator logs (Appendix C.6 log format): storages, views, multi-output and
# in-place operators, explicit reference counting
# ----------------------------------------------------------------------------

LOG_MEMORY, LOG_ALIAS, LOG_CALL, LOG_MUTATE, LOG_CONSTANT, LOG_COPY, LOG_COPYFROM, LOG_RELEASE = range(8)
LOG_KIND_NAMES = ["MEMORY", "ALIAS", "CALL", "MUTATE", "CONSTANT", "COPY", "COPYFROM", "RELEASE"]


@dataclass
class Log:
    """A log as parallel arrays, one row per instruction.  Names are integers.
      MEMORY   a = name, value = size          ALIAS    a = name, b = viewed name or -1
      CALL     ids = inputs then outputs (n_in inputs), value = cost; each output
               is then described by MEMORY and ALIAS, in output order
      MUTATE   ids = inputs then mutated inputs (n_in inputs), value = cost
      CONSTANT a = name (then MEMORY)           COPY     a = new name, b = name
      COPYFROM a = name, b = name               RELEASE  a = name"""
    name: str
    kind: np.ndarray              # int32 [n]
    a: np.ndarray                 # int32 [n]
    b: np.ndarray                 # int32 [n]
    n_in: np.ndarray              # int32 [n]
    value: np.ndarray             # int64 [n]
    list_offsets: np.ndarray      # int64 [n + 1]
    ids: np.ndarray               # int32 [list_offsets[n]]
    n_names: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def n_instrs(self) -> int:
        return int(self.kind.shape[0])

    def lists(self, i: int):
        lo, hi = int(self.list_offsets[i]), int(self.list_offsets[i + 1])
        k = int(self.n_in[i])
        return self.ids[lo:lo + k], self.ids[lo + k:hi]

    def digest(self) -> str:
        h = hashlib.sha256()
        for arr in (self.kind, self.a, self.b, self.n_in, self.value, self.list_offsets, self.ids):
            h.update(np.ascontiguousarray(arr).tobytes())
        return h.hexdigest()


class LogBuilder:
    def __init__(self, name: str):
        self.name = name
        self.rows = []            # (kind, a, b, n_in, value, ids)
        self.next_name = 0

    def fresh(self) -> int:
        self.next_name += 1
        return self.next_name - 1

    def _row(self, kind, a=-1, b=-1, value=0, ins=(), outs=()):
        self.rows.append((kind, a, b, len(ins), value, list(ins) + list(outs)))

    def constant(self, t, size):
        self._row(LOG_CONSTANT, a=t)
        self._row(LOG_MEMORY, a=t, value=size)

    def call(self, ins, outs, cost, sizes, aliases):
        """outs[k] has MEMORY sizes[k] and ALIAS aliases[k] (a name or -1)."""
        self._row(LOG_CALL, value=cost, ins=ins, outs=outs)
        for o, sz, al in zip(outs, sizes, aliases):
            self._row(LOG_MEMORY, a=o, value=sz)
            self._row(LOG_ALIAS, a=o, b=al)

    def mutate(self, ins, muts, cost):
        self._row(LOG_MUTATE, value=cost, ins=ins, outs=muts)

    def copy(self, to, ti):
        self._row(LOG_COPY, a=to, b=ti)

    def copyfrom(self, to, ti):
        self._row(LOG_COPYFROM, a=to, b=ti)

    def release(self, t):
        self._row(LOG_RELEASE, a=t)

    def build(self, **meta) -> Log:
        n = len(self.rows)
        lens = [len(r[5]) for r in self.rows]
        off = np.zeros(n + 1, np.int64)
        off[1:] = np.cumsum(lens)
        ids = np.array([v for r in self.rows for v in r[5]], np.int32)
        return Log(self.name, np.array([r[0] for r in self.rows], np.int32),
                   np.array([r[1] for r in self.rows], np.int32), np.array([r[2] for r in self.rows], np.int32),
                   np.array([r[3] for r in self.rows], np.int32), np.array([r[4] for r in self.rows], np.int64),
                   off, ids, self.next_name, dict(meta))


def log_from_trace(tr: Trace) -> Log:
    """The trace as a log: constants first (CONSTANT, MEMORY), then one CALL per
    operation creating a fresh storage, and a RELEASE after the last reader of
    every tensor that is not a required output (after its producer if nothing
    reads it; constants that nothing reads are never released).  Names are the
    trace's tensor ids."""
    n, F = tr.n_tensors, tr.n_ops
    b = LogBuilder(tr.name + "-log")
    b.next_name = n
    last = np.full(n, -1, np.int64)
    prod = np.full(n, -1, np.int64)
    prod[tr.op_output] = np.arange(F)
    for o in range(F):
        for u in tr.inputs(o):
            last[u] = max(last[u], o)
    last = np.maximum(last, prod)
    rel = [[] for _ in range(F)]
    for t in range(n):
        if not (tr.tensor_flags[t] & FLAG_REQUIRED) and last[t] >= 0:
            rel[last[t]].append(t)
    for t in range(n):
        if tr.tensor_flags[t] & FLAG_CONSTANT:
            b.constant(t, int(tr.tensor_size[t]))
    for o in range(F):
        t = int(tr.op_output[o])
        b.call([int(u) for u in tr.inputs(o)], [t], int(tr.op_cost[o]), [int(tr.tensor_size[t])], [-1])
        for r in rel[o]:
            b.release(r)
    return b.build()


def log_peak(log: Log) -> int:
    """Peak memory of a log replayed with no eviction: each operator adds its
    new storages, and a storage whose last reference goes is freed after the
    operator it follows (constants stay).  The log's own memory profile, used
    to space budgets."""
    name = {}                      # name -> storage
    size, const, refs = [], [], []
    mem = peak = 0
    pending = []                   # storages released since the last operator

    def drop(st):
        refs[st] -= 1
        if refs[st] == 0:
            pending.append(st)

    def flush():
        nonlocal mem
        for st in pending:
            if not const[st]:
                mem -= size[st]
        pending.clear()

    def new(sz, c):
        size.append(sz)
        const.append(c)
        refs.append(0)
        return len(size) - 1

    i, n = 0, log.n_instrs
    while i < n:
        k = int(log.kind[i])
        if k == LOG_CONSTANT:
            flush()
            st = new(int(log.value[i + 1]), True)
            mem += size[st]
            peak = max(peak, mem)
            name[int(log.a[i])] = st
            refs[st] += 1
            i += 2
        elif k == LOG_CALL:
            flush()
            ins, outs = log.lists(i)
            need, bound = 0, []
            own = {}
            for j, o in enumerate(outs):
                al = int(log.b[i + 2 + 2 * j])
                if al < 0:
                    st = new(int(log.value[i + 1 + 2 * j]), False)
                    need += size[st]
                    own[int(o)] = st
                else:
                    st = own[al] if al in own else name[al]
                bound.append((int(o), st))
            mem += need
            peak = max(peak, mem)
            for o, st in bound:
                name[o] = st
                refs[st] += 1
            i += 1 + 2 * len(outs)
        elif k == LOG_MUTATE:
            flush()
            _, muts = log.lists(i)
            clones = [new(size[name[int(m)]], False) for m in muts]
            mem += sum(size[c] for c in clones)
            peak = max(peak, mem)
            for m, c in zip(muts, clones):
                old = name[int(m)]
                name[int(m)] = c
                refs[c] += 1
                drop(old)
            i += 1
        elif k == LOG_COPY:
            name[int(log.a[i])] = name[int(log.b[i])]
            refs[name[int(log.b[i])]] += 1
            i += 1
        elif k == LOG_COPYFROM:
            old = name[int(log.a[i])]
            name[int(log.a[i])] = name[int(log.b[i])]
            refs[name[int(log.b[i])]] += 1
            drop(old)
            i += 1
        elif k == LOG_RELEASE:
            drop(name.pop(int(log.a[i])))
            i += 1
        else:
            raise ValueError(f"instruction {i}: unexpected kind {k}")
    return int(peak)


def resnet_log(seed: int = 2, blocks: int = 50) -> Log:
    """A PyTorch-style log of one training step of a ResNet-like network, as
    the DTR prototype records it: weights are constants; batch norm is one
    call with three outputs (result, saved mean, saved inverse std); ReLU is
    in place (MUTATE); autograd keeps saved tensors as extra references (COPY)
    dropped when their backward operator has run (RELEASE); the head flattens
    through a view; the backward pass computes input and weight gradients in
    one call, passes the residual gradient by reference and accumulates it,
    and keeps every weight gradient and the loss to the end.  Activation sizes
    are log-normal (median 4 MiB, sigma 1), weights log-normal (median 1 MiB,
    sigma 0.5); every cost is max(1, bytes // 4096) x U{1..4}."""
    rng = np.random.Generator(np.random.PCG64(seed))
    b = LogBuilder(f"resnet{blocks}-log")
    size = {}

    def act():
        return max(1, int(round(rng.lognormal(math.log(4 * MiB), 1.0))))

    def cost(nbytes):
        return max(1, nbytes // 4096) * int(rng.integers(1, 5))

    def const(nbytes):
        t = b.fresh()
        b.constant(t, nbytes)
        size[t] = nbytes
        return t

    def call(ins, sizes, aliases=None):
        outs = [b.fresh() for _ in sizes]
        aliases = aliases if aliases is not None else [-1] * len(sizes)
        own = sum(sz for sz, al in zip(sizes, aliases) if al < 0)
        b.call(ins, outs, cost(max(own, 1)) if own else 1, sizes, aliases)
        for o, sz, al in zip(outs, sizes, aliases):
            size[o] = size[al] if al >= 0 else sz
        return outs

    def relu_(t):
        b.mutate([t], [t], cost(size[t]))

    def save(t):
        c = b.fresh()
        b.copy(c, t)
        size[c] = size[t]
        return c

    def drop(*ts):
        for t in ts:
            b.release(t)

    STAT = 4096
    keep = []
    x, = call([], [act()])                          # the input batch
    tape = []
    for _ in range(blocks):
        w1, w2 = (const(max(1, int(round(rng.lognormal(math.log(MiB), 0.5))))) for _ in range(2))
        g1, g2 = const(STAT), const(STAT)
        sv = dict(w1=w1, w2=w2, g1=g1, g2=g2, x=save(x))
        y1, = call([x, w1], [act()])
        z1, m1, v1 = call([y1, g1], [size[y1], STAT, STAT])
        sv.update(y1=save(y1), m1=save(m1), v1=save(v1))
        drop(y1, m1, v1)
        relu_(z1)
        sv["z1"] = save(z1)
        y2, = call([z1, w2], [act()])
        drop(z1)
        z2, m2, v2 = call([y2, g2], [size[y2], STAT, STAT])
        sv.update(y2=save(y2), m2=save(m2), v2=save(v2))
        drop(y2, m2, v2)
        s, = call([z2, x], [size[z2]])
        drop(z2, x)
        relu_(s)
        sv["s"] = save(s)
        tape.append(sv)
        x = s
    wfc = const(4 * 2048 * 1000)
    f, = call([x], [size[x]], [x])                  # flatten: a view
    drop(x)
    logits, = call([f, wfc], [4 * 64 * 1000])
    sf, sl = save(f), save(logits)
    drop(f)
    loss, = call([logits], [4])
    drop(logits)
    keep.append(loss)
    # backward
    gl, = call([loss], [4])
    glog, = call([gl, sl], [size[sl]])
    drop(gl, sl)
    gf, gwfc = call([glog, sf, wfc], [size[sf], size[wfc]])
    drop(glog, sf)
    keep.append(gwfc)
    g, = call([gf], [size[gf]], [gf])               # unflatten the gradient: a view
    drop(gf)
    for sv in reversed(tape):
        ga, = call([g, sv["s"]], [size[sv["s"]]])    # ReLU backward from its output
        drop(g, sv["s"])
        gskip = save(ga)                            # the residual branch shares the gradient
        gy2, gg2 = call([ga, sv["y2"], sv["g2"], sv["m2"], sv["v2"]], [size[sv["y2"]], STAT])
        drop(ga, sv["y2"], sv["m2"], sv["v2"])
        gz1, gw2 = call([gy2, sv["z1"], sv["w2"]], [size[sv["z1"]], size[sv["w2"]]])
        drop(gy2)
        gz1r, = call([gz1, sv["z1"]], [size[sv["z1"]]])
        drop(gz1, sv["z1"])
        gy1, gg1 = call([gz1r, sv["y1"], sv["g1"], sv["m1"], sv["v1"]], [size[sv["y1"]], STAT])
        drop(gz1r, sv["y1"], sv["m1"], sv["v1"])
        gx1, gw1 = call([gy1, sv["x"], sv["w1"]], [size[sv["x"]], size[sv["w1"]]])
        drop(gy1, sv["x"])
        g, = call([gx1, gskip], [size[gx1]])        # gradient accumulation at the block input
        drop(gx1, gskip)
        keep += [gg2, gw2, gg1, gw1]
    keep.append(g)
    return b.build(seed=seed, blocks=blocks, kept=len(keep))


def config_resnet_log(blocks: int = 50) -> Workload:
    """The ResNet log at 256 budgets from 10% to 100% of its no-eviction peak
    x {h_DTR, h_DTR^eq, h_DTR^local, h_LRU, h_size, h_rand}: 1536 replays."""
    lg = resnet_log(blocks=blocks)
    peak = log_peak(lg)
    rows = []
    for h in (H_DTR, H_EQ, H_LOCAL, H_LRU, H_SIZE, H_RAND):
        for bud in linear_budgets(peak, 10, 100, 256):
            rows.append((0, h, bud, 2 * (1 << 32) + len(rows)))
    return Workload(f"resnet{blocks}log", [lg], _specs(rows), [peak],
                    f"PyTorch-style ResNet log, {blocks} blocks, 256 budgets x 6 heuristics")


CONFIGS["resnet50log"] = config_resnet_log


def random_log(seed: int, n_steps: int, n_const: int = 3, max_size: int = 8, max_cost: int = 5,
               max_in: int = 3, keep: int = 2) -> Log:
    """A PyTorch-like random log: constants; operator calls whose outputs are
    fresh storages or views of an input (or of an earlier output of the same
    call), with 1-3 outputs; in-place operators; variable copies and
    rebindings; releases of dead variables.  At the end every name but `keep`
    of them is released, so those stay live (the output condition)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    b = LogBuilder(f"randlog{seed}")
    live = []
    for _ in range(n_const):
        t = b.fresh()
        b.constant(t, int(rng.integers(1, max_size + 1)))
        live.append(t)
    for _ in range(n_steps):
        r = rng.random()
        if not live or r < 0.5:
            k = int(rng.integers(0, min(max_in, len(live)) + 1))
            ins = [live[int(i)] for i in rng.choice(len(live), size=k, replace=False)] if k else []
            n_out = 1 if rng.random() < 0.75 else int(rng.integers(2, 4))
            outs, sizes, aliases, roots = [], [], [], []
            for j in range(n_out):
                o = b.fresh()
                view = (ins or roots) and rng.random() < 0.3
                if view:
                    pool = ins + roots
                    aliases.append(pool[int(rng.integers(0, len(pool)))])
                else:
                    aliases.append(-1)
                    roots.append(o)
                outs.append(o)
                sizes.append(int(rng.integers(1, max_size + 1)))
            cost = 1 if all(a >= 0 for a in aliases) else int(rng.integers(1, max_cost + 1))
            b.call(ins, outs, cost, sizes, aliases)
            live += outs
        elif r < 0.62:
            k = int(rng.integers(1, min(max_in, len(live)) + 1))
            ins = [live[int(i)] for i in rng.choice(len(live), size=k, replace=False)]
            b.mutate(ins, [ins[0]], int(rng.integers(1, max_cost + 1)))
        elif r < 0.68:
            to = b.fresh()
            b.copy(to, live[int(rng.integers(0, len(live)))])
            live.append(to)
        elif r < 0.72 and len(live) >= 2:
            i, j = rng.choice(len(live), size=2, replace=False)
            b.copyfrom(live[int(i)], live[int(j)])
        else:
            i = int(rng.integers(0, len(live)))
            b.release(live.pop(i))
    order = rng.permutation(len(live))
    for i in order[keep:]:
        b.release(live[int(i)])
    return b.build(seed=seed)
