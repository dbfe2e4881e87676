/*
 * dtr_oracle.c -- plain, slow, CPU reference of Dynamic Tensor
 * Rematerialization's greedy eviction loop (Kirisame et al., ICLR 2021).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU path; the two meet only in the input
 * arrays produced by the workload generators.
 *
 * What it computes, step by step in the paper's order:
 *   - operator call (Section 2, Figure 1 prose; Appendix C.4
 *     "(Re)materialization"): lock every input, rematerialize evicted inputs
 *     recursively through their parent operation, allocate the output
 *     (evicting while memory is insufficient), advance the clock by the
 *     operator cost, unlock;
 *   - eviction (Appendix C.4 "Eviction and banishing"): the evictable pool is
 *     resident storages with no locks (Appendix C.1); the lowest score is
 *     evicted (Appendix C.4 "Runtime state");
 *   - deallocation policies (Section 2 "Deallocation"; Appendix C.4
 *     "Eviction and banishing"; Appendix C.5 "Banishing and eager eviction";
 *     compared in Appendix D): eager eviction of a released tensor, ignoring
 *     releases, or banishing -- a released tensor with no evicted child is
 *     removed for good (constants included) and its children are pinned
 *     (never evictable again); otherwise it is retried whenever one of its
 *     children is rematerialized;
 *   - heuristics of Section 4.1 and Appendix C.3: h_DTR with the exact
 *     evicted neighbourhood e* (Appendix C.2), h_DTR^eq with the union-find
 *     relaxation and its split approximation (Appendix C.2), h_DTR^local,
 *     h_LRU, h_size, h_rand, h_MSPS (cost of the evicted ancestors e_R over
 *     size, Section 4.1); h_{e*} of Appendix A.3 (no staleness); and the
 *     ablation family h'(s, m, c) = c / (m * s) of Appendix D, with staleness
 *     s and size m each used or not, and c the full e* cost, the
 *     equivalence-class cost, the local cost or none (c = 1);
 *   - output condition: tensors the program still holds at the end are
 *     rematerialized and locked (Appendix C.6 log semantics);
 *   - the prototype's search approximations (Appendix E): candidates smaller
 *     than 1% of the pool's mean size are ignored, and/or only a random
 *     sample of the pool is searched (each candidate kept with probability
 *     ceil(sqrt(n))/n); when nothing is left the search falls back to every
 *     candidate that is not small.
 *
 * No caching, no incremental data structure beyond the paper's own
 * union-find: every eviction rescans every tensor and every h_DTR score
 * walks its evicted neighbourhood from scratch.  Native recursion.
 *
 * Readings where the paper is silent (each is also a documented design
 * decision of the build): ties on score go to the smaller tensor id; the
 * clock is in integer cost units and last_access is stamped before the clock
 * advances, so staleness is >= 1 for every candidate; the pool excludes
 * constants; dead (released) tensors stay in the graph as evicted nodes and
 * count in e* and in union-find components; h_rand draws a fresh 64-bit
 * value per (seed, budget-eviction number, tensor id) from the SplitMix64
 * finaliser; the clock guard stops a simulation once the clock reaches 2^40.
 *
 * All quantities are integers; scores N/D are compared exactly by 128-bit
 * cross-multiplication.
 */
#define _GNU_SOURCE
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <pthread.h>

#define O_FLAG_CONSTANT 1u
#define O_FLAG_REQUIRED 2u

enum { ST_UNCOMPUTED = 0, ST_RESIDENT = 1, ST_EVICTED = 2, ST_BANISHED = 3 };
enum { OP_EAGER = 0, OP_IGNORE = 1, OP_BANISH = 2 };   /* deallocation policies */
enum { OH_DTR = 0, OH_EQ = 1, OH_LOCAL = 2, OH_LRU = 3, OH_SIZE = 4, OH_RAND = 5, OH_ESTAR = 6, OH_MSPS = 7,
       OH_FAMILY = 16 /* h'(s, m, c): 16 + 4c + 2s + m, s and m 1 = used */ };
enum { OC_ESTAR = 0, OC_EQCLASS = 1, OC_LOCAL = 2, OC_NONE = 3 };

static int family(int h) { return h >= OH_FAMILY && h < OH_FAMILY + 16; }
static int family_c(int h) { return (h - OH_FAMILY) >> 2; }
/* heuristics that keep the union-find components of Appendix C.2 */
static int uses_uf(int h) { return h == OH_EQ || (family(h) && family_c(h) == OC_EQCLASS); }
enum { OS_OK = 0, OS_OOM = 1, OS_CLOCK_OVERFLOW = 2, OS_STOPPED = 100 };

#define CLOCK_LIMIT ((int64_t)1 << 40)

typedef unsigned __int128 u128;

/* one trace, as handed over by the caller (arrays are borrowed) */
typedef struct {
    int32_t n_tensors, n_ops;
    const int64_t *tensor_size;
    const uint8_t *tensor_flags;
    const int32_t *op_output;
    const int64_t *op_cost;
    const int64_t *op_input_offsets;
    const int32_t *op_inputs;
} oracle_trace;

typedef struct { int32_t trace, heuristic; int64_t budget; uint64_t seed; int32_t policy, search; } oracle_spec;
enum { OSR_IGNORE_SMALL = 1, OSR_SAMPLE = 2 };   /* search approximation flags */

/* result fields (int64 each) */
enum {
    R_TOTAL_COST, R_BASE_COST, R_REMAT_COST, R_PEAK, R_FINAL_MEM, R_EXECUTED, R_REMATS,
    R_EVICTIONS, R_EAGER, R_SCORES, R_NBR_VISITS, R_ADJ_VISITS, R_STATUS, R_FAILED_OP, R_NFIELDS
};

/* optional probes used by tests */
typedef struct {
    int64_t stop_after_op;        /* >=0: stop once this op (incl. its releases) is done */
    int64_t stop_at_eviction;     /* >=0: stop at the start of this budget-eviction decision */
    uint8_t *state_out;           /* [n_tensors] state at the stop point (or at the end) */
    int32_t *locks_out;           /* [n_tensors] */
    int64_t *last_out;            /* [n_tensors] */
    uint64_t *score_n_out;        /* [n_tensors] N of each candidate at stop_at_eviction */
    uint64_t *score_d_lo_out;     /* [n_tensors] low 64 bits of D */
    uint64_t *score_d_hi_out;     /* [n_tensors] high 64 bits of D */
    uint8_t *candidate_out;       /* [n_tensors] 1 if in the pool at stop_at_eviction */
    int64_t *clock_out;           /* [1] clock at the stop point */
    int32_t *evict_log;           /* budget-evicted ids in order */
    int64_t evict_log_cap;
    int64_t *evict_log_len;
    int32_t *remat_log;           /* rematerialized ids in order */
    int64_t remat_log_cap;
    int64_t *remat_log_len;
    int64_t *uf_cost_sum_out;     /* [1] sum of running costs over union-find roots */
} oracle_probe;

/* ---------------------------------------------------------------- graph -- */

typedef struct {
    const oracle_trace *tr;
    int32_t *producer;       /* op producing tensor t, -1 for constants            */
    int64_t *c0;             /* cost of the producing op (0 for constants)         */
    int64_t *ch_off;         /* children(t): outputs of ops that read t            */
    int32_t *ch;
    int64_t *rel_off;        /* tensors released after op o, ascending id          */
    int32_t *rel;
} graph;

static void graph_free(graph *g)
{
    free(g->producer); free(g->c0); free(g->ch_off); free(g->ch); free(g->rel_off); free(g->rel);
}

/* parents(t) = inputs of t's parent operation (Appendix C.2 "Data dependencies");
 * children(t) = tensors whose parent operation reads t (the dependents, deps^T);
 * a tensor whose last external reference goes away after op o is released
 * after o (reference counting, Appendix A.2) unless it is a required output;
 * a constant is released after its last reader (one that nothing reads is
 * never released). */
static int graph_build(graph *g, const oracle_trace *tr)
{
    int32_t n = tr->n_tensors, F = tr->n_ops;
    memset(g, 0, sizeof(*g));
    g->tr = tr;
    g->producer = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    g->c0 = calloc((size_t)(n > 0 ? n : 1), sizeof(int64_t));
    g->ch_off = calloc((size_t)n + 1, sizeof(int64_t));
    g->rel_off = calloc((size_t)F + 1, sizeof(int64_t));
    int64_t E = tr->op_input_offsets[F];
    g->ch = malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
    g->rel = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
    int64_t *last = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *fill = malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!g->producer || !g->c0 || !g->ch_off || !g->rel_off || !g->ch || !g->rel || !last || !fill) {
        free(last); free(fill); graph_free(g); return -1;
    }
    for (int32_t t = 0; t < n; t++) { g->producer[t] = -1; last[t] = -1; }
    for (int32_t o = 0; o < F; o++) {
        int32_t t = tr->op_output[o];
        g->producer[t] = o;
        g->c0[t] = tr->op_cost[o];
        if (last[t] < o) last[t] = o;
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++) {
            int32_t u = tr->op_inputs[e];
            g->ch_off[u + 1]++;
            if (last[u] < o) last[u] = o;
        }
    }
    for (int32_t t = 0; t < n; t++) g->ch_off[t + 1] += g->ch_off[t];
    for (int32_t t = 0; t < n; t++) fill[t] = g->ch_off[t];
    for (int32_t o = 0; o < F; o++)
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++) {
            int32_t u = tr->op_inputs[e];
            g->ch[fill[u]++] = tr->op_output[o];
        }
    /* release lists: ascending id within an op */
    for (int32_t t = 0; t < n; t++) {
        if (tr->tensor_flags[t] & O_FLAG_REQUIRED) continue;
        if (last[t] >= 0) g->rel_off[last[t] + 1]++;
    }
    for (int32_t o = 0; o < F; o++) g->rel_off[o + 1] += g->rel_off[o];
    int64_t *rfill = malloc(sizeof(int64_t) * (size_t)(F > 0 ? F : 1));
    if (!rfill) { free(last); free(fill); graph_free(g); return -1; }
    for (int32_t o = 0; o < F; o++) rfill[o] = g->rel_off[o];
    for (int32_t t = 0; t < n; t++) {   /* ascending t gives ascending ids per list */
        if (tr->tensor_flags[t] & O_FLAG_REQUIRED) continue;
        if (last[t] >= 0) g->rel[rfill[last[t]]++] = t;
    }
    free(rfill); free(last); free(fill);
    return 0;
}

/* ------------------------------------------------------------ simulator -- */

typedef struct sim sim;

/* How the simulator sees the dependency graph: parents and children of a
 * node and its local cost c0, and what banishing a released node does.  A
 * trace has the static graph of its operators (below); the log section
 * supplies the storage graph of a replay, which grows as operators first
 * run. */
typedef struct {
    int64_t (*n_par)(const sim *s, int32_t u);
    int32_t (*par_at)(const sim *s, int32_t u, int64_t k);
    int64_t (*n_ch)(const sim *s, int32_t u);
    int32_t (*ch_at)(const sim *s, int32_t u, int64_t k);
    int64_t (*c0_of)(const sim *s, int32_t u);
    void (*try_banish)(sim *s, int32_t t);
} graph_view;

struct sim {
    const graph *g;
    const graph_view *view;
    const oracle_trace *tr;
    int heuristic;
    int policy;
    int search;                   /* OSR_* flags */
    int64_t budget;
    uint64_t seed;

    uint8_t *state;
    int32_t *locks;
    uint8_t *pinned;              /* children of banished tensors: never evictable */
    uint8_t *pending;             /* released, banishing deferred */
    int64_t *last_access;
    int64_t clock, memory, peak;
    int64_t r[R_NFIELDS];
    int64_t eviction_no;          /* budget evictions so far (h_rand key) */
    int stopped;
    int64_t cur_op;

    /* union-find over evicted components (h_DTR^eq), Appendix C.2 */
    int32_t *node_of;             /* current UF node of each tensor     */
    int32_t *uf_parent;
    int64_t *uf_cost;
    int64_t *uf_mark;             /* epoch stamps per UF node (root dedup) */
    int64_t uf_n, uf_cap;

    /* log replay: residency generation per storage, generation at which each
     * tensor's operator last ran (NULL for plain traces) */
    int64_t *sgen, *gen;
    const void *logp;             /* the lowered log (log replay only) */
    /* log replay: the storage graph as of now (Appendix C.2: indexed by time),
     * grown when an operator first creates its tensors */
    int64_t *dc0;                 /* cost of each storage's tensors created so far */
    int32_t **dpar, **dch;        /* parents and children created so far */
    int64_t *npar, *nch, *cpar, *cch;   /* their counts and capacities */

    /* scratch for neighbourhood walks */
    int64_t *mark;                /* epoch stamps */
    int64_t epoch;
    int32_t *queue;

    oracle_probe *probe;
};

static int32_t uf_new(sim *s)
{
    if (s->uf_n == s->uf_cap) {
        int64_t cap = s->uf_cap ? 2 * s->uf_cap : 1024;
        int32_t *p = realloc(s->uf_parent, sizeof(int32_t) * (size_t)cap);
        if (!p) return -1;
        s->uf_parent = p;
        int64_t *c = realloc(s->uf_cost, sizeof(int64_t) * (size_t)cap);
        if (!c) return -1;
        s->uf_cost = c;
        int64_t *m = realloc(s->uf_mark, sizeof(int64_t) * (size_t)cap);
        if (!m) return -1;
        memset(m + s->uf_cap, 0, sizeof(int64_t) * (size_t)(cap - s->uf_cap));
        s->uf_mark = m;
        s->uf_cap = cap;
    }
    int32_t id = (int32_t)s->uf_n++;
    s->uf_parent[id] = id;
    s->uf_cost[id] = 0;
    return id;
}

static int32_t uf_find(sim *s, int32_t x)
{
    int32_t root = x;
    while (s->uf_parent[root] != root) root = s->uf_parent[root];
    while (s->uf_parent[x] != root) {          /* path compression */
        int32_t next = s->uf_parent[x];
        s->uf_parent[x] = root;
        x = next;
    }
    return root;
}

static int32_t uf_union(sim *s, int32_t a, int32_t b)
{
    a = uf_find(s, a);
    b = uf_find(s, b);
    if (a == b) return a;
    s->uf_parent[b] = a;
    s->uf_cost[a] += s->uf_cost[b];
    return a;
}

static void evict(sim *s, int32_t v, int eager);

/* a banished tensor is never read again (its children are pinned), so a lock
 * on one means the policy's invariant broke */
static void lock(sim *s, int32_t t)
{
    if (s->state[t] == ST_BANISHED) abort();
    s->locks[t]++;
}
static void unlock(sim *s, int32_t t) { s->locks[t]--; }

static int is_evictable(const sim *s, int32_t t)
{
    return s->state[t] == ST_RESIDENT && s->locks[t] == 0 && !s->pinned[t] &&
           !(s->tr->tensor_flags[t] & O_FLAG_CONSTANT);
}

/* Banish t if none of its children is evicted and no operation in progress
 * holds it (Appendix C.4): its memory is reclaimed if resident, it leaves the
 * graph for good, and every resident child is pinned.  Otherwise t stays
 * pending and is retried when one of its children is rematerialized. */
static void trace_try_banish(sim *s, int32_t t)
{
    const graph *g = s->g;
    int blocked = s->locks[t] > 0;
    for (int64_t e = g->ch_off[t]; e < g->ch_off[t + 1] && !blocked; e++)
        if (s->state[g->ch[e]] == ST_EVICTED) blocked = 1;
    if (blocked) { s->pending[t] = 1; return; }
    s->pending[t] = 0;
    if (s->state[t] == ST_RESIDENT) s->memory -= s->tr->tensor_size[t];
    s->state[t] = ST_BANISHED;
    s->r[R_EAGER]++;              /* deallocation-driven removals */
    for (int64_t e = g->ch_off[t]; e < g->ch_off[t + 1]; e++)
        if (s->state[g->ch[e]] == ST_RESIDENT) s->pinned[g->ch[e]] = 1;
}

/* A trace's graph is static: the parents of u are the inputs of its parent
 * operation, its children the outputs of the operations reading u, its cost
 * c0 that of its parent operation. */
static int64_t trace_n_par(const sim *s, int32_t u)
{
    int32_t o = s->g->producer[u];
    return o < 0 ? 0 : s->tr->op_input_offsets[o + 1] - s->tr->op_input_offsets[o];
}
static int32_t trace_par_at(const sim *s, int32_t u, int64_t k)
{
    return s->tr->op_inputs[s->tr->op_input_offsets[s->g->producer[u]] + k];
}
static int64_t trace_n_ch(const sim *s, int32_t u) { return s->g->ch_off[u + 1] - s->g->ch_off[u]; }
static int32_t trace_ch_at(const sim *s, int32_t u, int64_t k) { return s->g->ch[s->g->ch_off[u] + k]; }
static int64_t trace_c0_of(const sim *s, int32_t u) { return s->g->c0[u]; }

static const graph_view TRACE_VIEW = {trace_n_par, trace_par_at, trace_n_ch, trace_ch_at, trace_c0_of,
                                      trace_try_banish};

/* the graph as the current simulation sees it */
static int64_t n_par(const sim *s, int32_t u) { return s->view->n_par(s, u); }
static int32_t par_at(const sim *s, int32_t u, int64_t k) { return s->view->par_at(s, u, k); }
static int64_t n_ch(const sim *s, int32_t u) { return s->view->n_ch(s, u); }
static int32_t ch_at(const sim *s, int32_t u, int64_t k) { return s->view->ch_at(s, u, k); }
static int64_t c0_of(const sim *s, int32_t u) { return s->view->c0_of(s, u); }
static void try_banish(sim *s, int32_t t) { s->view->try_banish(s, t); }

/* deallocation of t after its last reader (Section 2, Appendix C.5) */
static void release(sim *s, int32_t t)
{
    if (s->policy == OP_EAGER) {
        if (is_evictable(s, t)) evict(s, t, 1);
    } else if (s->policy == OP_BANISH) {
        try_banish(s, t);
    }
}

/* e_R(x) (Section 4.1): evicted tensors reachable from x through evicted
 * parents only, i.e. those that rematerializing x would rematerialize.
 * Returns the sum of their local costs; the set size goes to *count. */
static int64_t ancestors_cost(sim *s, int32_t x, int64_t *count)
{
    int64_t sum = 0, cnt = 0;
    s->epoch++;
    int64_t head = 0, tail = 0;
    s->queue[tail++] = x;
    while (head < tail) {
        int32_t u = s->queue[head++];
        for (int64_t k = 0; k < n_par(s, u); k++) {
            int32_t p = par_at(s, u, k);
            if (s->state[p] != ST_EVICTED || s->mark[p] == s->epoch) continue;
            s->mark[p] = s->epoch;
            sum += c0_of(s, p);
            cnt++;
            s->queue[tail++] = p;
        }
    }
    *count = cnt;
    return sum;
}

/* Exact evicted neighbourhood e*(x) (Appendix C.2): the evicted ancestors
 * e_R(x), together with the evicted tensors reachable from x through evicted
 * children only (descendants).  The two sets are disjoint (the graph is
 * acyclic).  Returns the sum of their local costs; the set size goes to
 * *count. */
static int64_t estar_cost(sim *s, int32_t x, int64_t *count)
{
    int64_t cnt = 0;
    int64_t sum = ancestors_cost(s, x, &cnt);
    /* descendants (same epoch: a tensor is never on both sides) */
    int64_t head = 0, tail = 0;
    s->queue[tail++] = x;
    while (head < tail) {
        int32_t u = s->queue[head++];
        for (int64_t k = 0; k < n_ch(s, u); k++) {
            int32_t c = ch_at(s, u, k);
            if (s->state[c] != ST_EVICTED || s->mark[c] == s->epoch) continue;
            s->mark[c] = s->epoch;
            sum += c0_of(s, c);
            cnt++;
            s->queue[tail++] = c;
        }
    }
    *count = cnt;
    return sum;
}

/* Relaxed neighbourhood cost (Appendix C.2): the union of the union-find sets
 * of x's evicted parents and evicted children, each distinct set counted once,
 * merged only for the query (no union is performed). */
static int64_t eq_cost(sim *s, int32_t x, int64_t *count)
{
    int64_t sum = 0, cnt = 0;
    s->epoch++;
    for (int64_t k = 0; k < n_par(s, x); k++) {
        int32_t p = par_at(s, x, k);
        if (s->state[p] != ST_EVICTED) continue;
        cnt++;
        int32_t r = uf_find(s, s->node_of[p]);
        if (s->uf_mark[r] == s->epoch) continue;
        s->uf_mark[r] = s->epoch;
        sum += s->uf_cost[r];
    }
    for (int64_t k = 0; k < n_ch(s, x); k++) {
        int32_t c = ch_at(s, x, k);
        if (s->state[c] != ST_EVICTED) continue;
        cnt++;
        int32_t r = uf_find(s, s->node_of[c]);
        if (s->uf_mark[r] == s->epoch) continue;
        s->uf_mark[r] = s->epoch;
        sum += s->uf_cost[r];
    }
    *count = cnt;
    return sum;
}

static int64_t degree(const sim *s, int32_t x) { return n_par(s, x) + n_ch(s, x); }

/* SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): state advanced by the
 * golden-ratio gamma, then the variant-13 output mix. */
static uint64_t splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* score N/D of candidate x (Section 4.1 and Appendix C.3; h_{e*} from A.3) */
static void score(sim *s, int32_t x, uint64_t *N, u128 *D)
{
    int64_t stale = s->clock - s->last_access[x];   /* >= 1 by construction */
    int64_t m = s->tr->tensor_size[x];
    int64_t c0 = c0_of(s, x);
    int64_t cnt = 0;
    if (stale < 1) abort();
    switch (s->heuristic) {
    case OH_DTR:
        *N = (uint64_t)(c0 + estar_cost(s, x, &cnt));
        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;
        s->r[R_NBR_VISITS] += cnt;
        s->r[R_ADJ_VISITS] += degree(s, x);
        break;
    case OH_ESTAR:
        *N = (uint64_t)(c0 + estar_cost(s, x, &cnt));
        *D = (u128)(uint64_t)m;
        s->r[R_NBR_VISITS] += cnt;
        s->r[R_ADJ_VISITS] += degree(s, x);
        break;
    case OH_EQ:
        *N = (uint64_t)(c0 + eq_cost(s, x, &cnt));
        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;
        s->r[R_NBR_VISITS] += cnt;
        s->r[R_ADJ_VISITS] += degree(s, x);
        break;
    case OH_LOCAL:
        *N = (uint64_t)c0;
        *D = (u128)(uint64_t)m * (u128)(uint64_t)stale;
        break;
    case OH_LRU:
        *N = 1;
        *D = (u128)(uint64_t)stale;
        break;
    case OH_SIZE:
        *N = 1;
        *D = (u128)(uint64_t)m;
        break;
    case OH_RAND: {
        uint64_t key = ((uint64_t)s->eviction_no << 32) + (uint64_t)(uint32_t)x;
        *N = splitmix64_mix(s->seed + 0x9E3779B97F4A7C15ull * key);
        *D = 1;
        break;
    }
    case OH_MSPS:
        *N = (uint64_t)(c0 + ancestors_cost(s, x, &cnt));
        *D = (u128)(uint64_t)m;
        s->r[R_NBR_VISITS] += cnt;
        s->r[R_ADJ_VISITS] += degree(s, x);
        break;
    default: {
        if (!family(s->heuristic)) abort();
        /* h'(s, m, c)(x) = c(x) / (m(x) * s(x)), an ablated measure being 1 */
        const int h = s->heuristic - OH_FAMILY;
        switch (h >> 2) {
        case OC_ESTAR:
            *N = (uint64_t)(c0 + estar_cost(s, x, &cnt));
            s->r[R_NBR_VISITS] += cnt;
            s->r[R_ADJ_VISITS] += degree(s, x);
            break;
        case OC_EQCLASS:
            *N = (uint64_t)(c0 + eq_cost(s, x, &cnt));
            s->r[R_NBR_VISITS] += cnt;
            s->r[R_ADJ_VISITS] += degree(s, x);
            break;
        case OC_LOCAL:
            *N = (uint64_t)c0;
            break;
        default:
            *N = 1;
            break;
        }
        *D = (u128)(uint64_t)((h & 1) ? m : 1) * (u128)(uint64_t)((h & 2) ? stale : 1);
        break;
    }
    }
}

/* a strictly better than b: N_a/D_a < N_b/D_b, ties to the smaller id */
static int better(uint64_t na, u128 da, int32_t ia, uint64_t nb, u128 db, int32_t ib)
{
    u128 l = (u128)na * db, r = (u128)nb * da;
    if (l != r) return l < r;
    return ia < ib;
}

static void evict(sim *s, int32_t v, int eager)
{
    s->state[v] = ST_EVICTED;
    s->memory -= s->tr->tensor_size[v];
    if (eager) s->r[R_EAGER]++;
    else s->r[R_EVICTIONS]++;
    if (uses_uf(s->heuristic)) {
        /* add c0(v) to its component, then union with every evicted neighbour */
        int32_t r = uf_find(s, s->node_of[v]);
        s->uf_cost[r] += c0_of(s, v);
        for (int64_t k = 0; k < n_par(s, v); k++) {
            int32_t p = par_at(s, v, k);
            if (s->state[p] == ST_EVICTED) r = uf_union(s, r, s->node_of[p]);
        }
        for (int64_t k = 0; k < n_ch(s, v); k++) {
            int32_t c = ch_at(s, v, k);
            if (s->state[c] == ST_EVICTED) r = uf_union(s, r, s->node_of[c]);
        }
    }
}

static void dump_state(sim *s)
{
    oracle_probe *p = s->probe;
    if (!p) return;
    int32_t n = s->tr->n_tensors;
    if (p->state_out) memcpy(p->state_out, s->state, (size_t)n);
    if (p->locks_out) memcpy(p->locks_out, s->locks, sizeof(int32_t) * (size_t)n);
    if (p->last_out) memcpy(p->last_out, s->last_access, sizeof(int64_t) * (size_t)n);
    if (p->clock_out) p->clock_out[0] = s->clock;
    if (p->uf_cost_sum_out) {
        int64_t sum = 0;
        for (int64_t i = 0; i < s->uf_n; i++)
            if (s->uf_parent[i] == (int32_t)i) sum += s->uf_cost[i];
        p->uf_cost_sum_out[0] = sum;
    }
}

/* smallest r with r * r >= n */
static uint64_t ceil_sqrt(uint64_t n)
{
    uint64_t r = 0;
    while (r * r < n) r++;
    return r;
}

/* the sampling draw of candidate x at an eviction decision: SplitMix64 on a
 * stream of its own (the seed offset by a fixed odd constant) */
static uint64_t sample_key(uint64_t seed, int64_t eviction_no, int32_t x)
{
    uint64_t key = ((uint64_t)eviction_no << 32) + (uint64_t)(uint32_t)x;
    return splitmix64_mix((seed ^ 0xD6E8FEB86659FD93ull) + 0x9E3779B97F4A7C15ull * key);
}

/* while memory is insufficient, evict the lowest-scored evictable tensor
 * (of the searched candidates, under the search approximations) */
static void allocate(sim *s, int64_t size)
{
    int32_t n = s->tr->n_tensors;
    while (s->memory + size > s->budget) {
        oracle_probe *p = s->probe;
        int dumping = p && p->stop_at_eviction >= 0 && s->eviction_no == p->stop_at_eviction;
        /* pool statistics for the approximations: count and total size */
        int64_t n0 = 0, size_sum = 0;
        for (int32_t x = 0; x < n; x++)
            if (is_evictable(s, x)) { n0++; size_sum += s->tr->tensor_size[x]; }
        /* sampling: keep each candidate with probability k/n0, k = ceil(sqrt(n0)) */
        uint64_t k = ceil_sqrt((uint64_t)n0);
        int sample_all = k >= (uint64_t)n0;
        uint64_t tau = sample_all ? 0 : (uint64_t)((((u128)k) << 64) / (u128)(uint64_t)n0);
        int32_t best = -1;
        uint64_t bn = 0;
        u128 bd = 0;
        int64_t count = 0;
        for (int pass = 0; pass < 2 && best < 0; pass++) {
            int sampling = pass == 0 && (s->search & OSR_SAMPLE) && !sample_all;
            if (pass == 1 && !(s->search & OSR_SAMPLE)) break;
            for (int32_t x = 0; x < n; x++) {
                if (!is_evictable(s, x)) continue;
                if ((s->search & OSR_IGNORE_SMALL) &&
                    (u128)100 * (u128)(uint64_t)s->tr->tensor_size[x] * (u128)(uint64_t)n0 < (u128)(uint64_t)size_sum)
                    continue;     /* smaller than 1% of the mean size */
                if (sampling && sample_key(s->seed, s->eviction_no, x) >= tau) continue;
                uint64_t N;
                u128 D;
                score(s, x, &N, &D);
                count++;
                if (dumping) {
                    if (p->score_n_out) p->score_n_out[x] = N;
                    if (p->score_d_lo_out) p->score_d_lo_out[x] = (uint64_t)D;
                    if (p->score_d_hi_out) p->score_d_hi_out[x] = (uint64_t)(D >> 64);
                    if (p->candidate_out) p->candidate_out[x] = 1;
                }
                if (best < 0 || better(N, D, x, bn, bd, best)) { best = x; bn = N; bd = D; }
            }
        }
        if (dumping) { dump_state(s); s->stopped = OS_STOPPED; s->r[R_STATUS] = OS_STOPPED; return; }
        if (best < 0) { s->r[R_STATUS] = OS_OOM; s->stopped = OS_OOM; return; }
        s->r[R_SCORES] += count;
        if (p && p->evict_log && *p->evict_log_len < p->evict_log_cap)
            p->evict_log[(*p->evict_log_len)++] = best;
        evict(s, best, 0);
        s->eviction_no++;
    }
}

/* run op o producing t: stamp last_access, advance the clock by the op cost */
static void execute(sim *s, int32_t o, int32_t t, int remat)
{
    const oracle_trace *tr = s->tr;
    for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
        s->last_access[tr->op_inputs[e]] = s->clock;
    s->last_access[t] = s->clock;
    int64_t c = tr->op_cost[o];
    s->clock += c;
    s->r[R_TOTAL_COST] += c;
    s->r[R_EXECUTED]++;
    if (remat) { s->r[R_REMATS]++; s->r[R_REMAT_COST] += c; }
    else s->r[R_BASE_COST] += c;
    s->memory += tr->tensor_size[t];
    if (s->memory > s->peak) s->peak = s->memory;
    s->state[t] = ST_RESIDENT;
    if (uses_uf(s->heuristic)) {
        if (remat) {
            /* split approximation: subtract c0 from the old set, move t to a fresh empty set */
            int32_t r = uf_find(s, s->node_of[t]);
            s->uf_cost[r] -= s->g->c0[t];
        }
        int32_t nd = uf_new(s);
        if (nd < 0) abort();
        s->node_of[t] = nd;
    }
    if (s->clock >= CLOCK_LIMIT) { s->r[R_STATUS] = OS_CLOCK_OVERFLOW; s->stopped = OS_CLOCK_OVERFLOW; }
}

/* rematerialize evicted u by replaying its parent operation (recursive) */
static void remat(sim *s, int32_t u)
{
    const oracle_trace *tr = s->tr;
    int32_t o = s->g->producer[u];
    oracle_probe *p = s->probe;
    if (p && p->remat_log && *p->remat_log_len < p->remat_log_cap)
        p->remat_log[(*p->remat_log_len)++] = u;
    for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
        lock(s, tr->op_inputs[e]);
    for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++) {
        int32_t q = tr->op_inputs[e];
        if (s->state[q] == ST_EVICTED) {
            remat(s, q);
            if (s->stopped) return;
        }
    }
    allocate(s, tr->tensor_size[u]);
    if (s->stopped) return;
    execute(s, o, u, 1);
    if (s->stopped) return;
    for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
        unlock(s, tr->op_inputs[e]);
    /* u is a dependent of each of its parents: retry their deferred banishing */
    if (s->policy == OP_BANISH)
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
            if (s->pending[tr->op_inputs[e]]) try_banish(s, tr->op_inputs[e]);
}

static void sim_run(sim *s)
{
    const oracle_trace *tr = s->tr;
    const graph *g = s->g;
    int32_t n = tr->n_tensors;
    s->r[R_FAILED_OP] = -1;
    s->cur_op = 0;
    /* constants: resident from time 0, never evictable */
    for (int32_t t = 0; t < n; t++) {
        if (!(tr->tensor_flags[t] & O_FLAG_CONSTANT)) continue;
        s->state[t] = ST_RESIDENT;
        s->memory += tr->tensor_size[t];
        if (s->memory > s->peak) s->peak = s->memory;
    }
    if (s->memory > s->budget) { s->r[R_STATUS] = OS_OOM; s->stopped = OS_OOM; goto done; }

    for (int32_t o = 0; o < tr->n_ops; o++) {
        s->cur_op = o;
        int32_t t = tr->op_output[o];
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
            lock(s, tr->op_inputs[e]);
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++) {
            int32_t u = tr->op_inputs[e];
            if (s->state[u] == ST_EVICTED) {
                remat(s, u);
                if (s->stopped) goto done;
            }
        }
        allocate(s, tr->tensor_size[t]);
        if (s->stopped) goto done;
        execute(s, o, t, 0);
        if (s->stopped) goto done;
        for (int64_t e = tr->op_input_offsets[o]; e < tr->op_input_offsets[o + 1]; e++)
            unlock(s, tr->op_inputs[e]);
        for (int64_t e = g->rel_off[o]; e < g->rel_off[o + 1]; e++) release(s, g->rel[e]);
        if (s->probe && s->probe->stop_after_op == o) {
            dump_state(s);
            s->stopped = OS_STOPPED;
            s->r[R_STATUS] = OS_STOPPED;
            goto done;
        }
    }
    /* output condition: every required output resident (and held) at the end */
    s->cur_op = tr->n_ops;
    for (int32_t t = 0; t < n; t++) {
        if (!(tr->tensor_flags[t] & O_FLAG_REQUIRED)) continue;
        lock(s, t);
        if (s->state[t] == ST_EVICTED) {
            remat(s, t);
            if (s->stopped) goto done;
        }
    }
    dump_state(s);
done:
    if (s->stopped == OS_OOM || s->stopped == OS_CLOCK_OVERFLOW) s->r[R_FAILED_OP] = s->cur_op;
    s->r[R_PEAK] = s->peak;
    s->r[R_FINAL_MEM] = s->memory;
}

static int run_one(const oracle_trace *tr, const graph *g, const oracle_spec *sp,
                   int64_t *result, oracle_probe *probe)
{
    int32_t n = tr->n_tensors;
    sim s;
    memset(&s, 0, sizeof(s));
    s.g = g;
    s.view = &TRACE_VIEW;
    s.tr = tr;
    s.heuristic = sp->heuristic;
    s.policy = sp->policy;
    s.search = sp->search;
    s.budget = sp->budget;
    s.seed = sp->seed;
    s.probe = probe;
    size_t nn = (size_t)(n > 0 ? n : 1);
    s.state = calloc(nn, 1);
    s.pinned = calloc(nn, 1);
    s.pending = calloc(nn, 1);
    s.locks = calloc(nn, sizeof(int32_t));
    s.last_access = calloc(nn, sizeof(int64_t));
    s.node_of = malloc(sizeof(int32_t) * nn);
    s.queue = malloc(sizeof(int32_t) * nn);
    s.mark = calloc(nn, sizeof(int64_t));
    int rc = 0;
    if (!s.state || !s.pinned || !s.pending || !s.locks || !s.last_access || !s.node_of || !s.queue || !s.mark)
        rc = -1;
    else {
        for (int32_t t = 0; t < n; t++) s.node_of[t] = -1;
        sim_run(&s);
        for (int i = 0; i < R_NFIELDS; i++) result[i] = s.r[i];
    }
    free(s.state); free(s.pinned); free(s.pending); free(s.locks); free(s.last_access); free(s.node_of);
    free(s.queue); free(s.mark);
    free(s.uf_parent); free(s.uf_cost); free(s.uf_mark);
    return rc;
}

/* ------------------------------------------------------------ public API -- */

/* Deep rematerialization chains recurse once per level, so every simulation
 * runs on a worker thread with a large stack. */
#define WORKER_STACK ((size_t)512 << 20)

typedef struct {
    const oracle_trace *traces;
    const graph *graphs;
    const oracle_spec *specs;
    int64_t *results;
    oracle_probe *probe;
    int32_t n_sims;
    int32_t next;                 /* shared cursor */
    pthread_mutex_t mu;
    int rc;
} batch;

static void *worker(void *arg)
{
    batch *b = arg;
    for (;;) {
        pthread_mutex_lock(&b->mu);
        int32_t i = b->next++;
        pthread_mutex_unlock(&b->mu);
        if (i >= b->n_sims) break;
        const oracle_spec *sp = &b->specs[i];
        int rc = run_one(&b->traces[sp->trace], &b->graphs[sp->trace], sp,
                         b->results + (int64_t)i * R_NFIELDS, b->probe);
        if (rc) { pthread_mutex_lock(&b->mu); b->rc = rc; pthread_mutex_unlock(&b->mu); }
    }
    return NULL;
}

int oracle_result_fields(void) { return R_NFIELDS; }

/* Run n_sims simulations over n_traces traces on n_threads threads.
 * results: int64 [n_sims * oracle_result_fields()].  probe may be NULL; with a
 * probe, n_sims must be 1.  Returns 0, or -1 on allocation failure, -2 on a
 * bad argument. */
int oracle_run(const oracle_trace *traces, int32_t n_traces, const oracle_spec *specs,
               int32_t n_sims, int64_t *results, int32_t n_threads, oracle_probe *probe)
{
    if (n_traces < 0 || n_sims < 0 || (probe && n_sims != 1)) return -2;
    for (int32_t i = 0; i < n_sims; i++)
        if (specs[i].trace < 0 || specs[i].trace >= n_traces ||
            !((specs[i].heuristic >= 0 && specs[i].heuristic <= OH_MSPS) || family(specs[i].heuristic)) ||
            specs[i].policy < OP_EAGER || specs[i].policy > OP_BANISH ||
            specs[i].search < 0 || specs[i].search > (OSR_IGNORE_SMALL | OSR_SAMPLE) ||
            (specs[i].policy == OP_BANISH && uses_uf(specs[i].heuristic)))
            return -2;
    graph *graphs = calloc((size_t)(n_traces > 0 ? n_traces : 1), sizeof(graph));
    if (!graphs) return -1;
    int rc = 0;
    int32_t built = 0;
    for (; built < n_traces; built++)
        if (graph_build(&graphs[built], &traces[built])) { rc = -1; break; }
    if (rc == 0) {
        batch b;
        memset(&b, 0, sizeof(b));
        b.traces = traces; b.graphs = graphs; b.specs = specs; b.results = results;
        b.probe = probe; b.n_sims = n_sims;
        pthread_mutex_init(&b.mu, NULL);
        if (n_threads < 1) n_threads = 1;
        if (n_threads > n_sims) n_threads = n_sims > 0 ? n_sims : 1;
        pthread_t *th = calloc((size_t)n_threads, sizeof(pthread_t));
        pthread_attr_t attr;
        pthread_attr_init(&attr);
        pthread_attr_setstacksize(&attr, WORKER_STACK);
        int started = 0;
        for (int i = 0; th && i < n_threads; i++)
            if (pthread_create(&th[i], &attr, worker, &b) == 0) started++;
        if (started == 0) rc = -1;
        for (int i = 0; i < started; i++) pthread_join(th[i], NULL);
        pthread_attr_destroy(&attr);
        pthread_mutex_destroy(&b.mu);
        free(th);
        if (b.rc) rc = b.rc;
    }
    for (int32_t i = 0; i < built; i++) graph_free(&graphs[i]);
    free(graphs);
    return rc;
}

/* Test hook: exact evicted-neighbourhood cost of x under a given state vector
 * (0 uncomputed, 1 resident, 2 evicted).  Returns sum of c0 over e*(x), or
 * over e_R(x) (the evicted ancestors only) when ancestors_only is set, and
 * writes the set size to *count and the membership to member_out (optional). */
int64_t oracle_estar(const oracle_trace *tr, const uint8_t *state, int32_t x, int64_t *count,
                     uint8_t *member_out, int32_t ancestors_only)
{
    graph g;
    if (graph_build(&g, tr)) return -1;
    sim s;
    memset(&s, 0, sizeof(s));
    s.g = &g;
    s.view = &TRACE_VIEW;
    s.tr = tr;
    size_t nn = (size_t)(tr->n_tensors > 0 ? tr->n_tensors : 1);
    s.state = malloc(nn);
    s.mark = calloc(nn, sizeof(int64_t));
    s.queue = malloc(sizeof(int32_t) * nn);
    int64_t sum = -1;
    if (s.state && s.mark && s.queue) {
        memcpy(s.state, state, (size_t)tr->n_tensors);
        sum = ancestors_only ? ancestors_cost(&s, x, count) : estar_cost(&s, x, count);
        if (member_out)
            for (int32_t t = 0; t < tr->n_tensors; t++) member_out[t] = (s.mark[t] == s.epoch);
    }
    free(s.state); free(s.mark); free(s.queue);
    graph_free(&g);
    return sum;
}

/* Test hook: the SplitMix64 draw used by h_rand for (seed, eviction number, id). */
uint64_t oracle_sample_key(uint64_t seed, int64_t eviction_no, int32_t x)
{
    return sample_key(seed, eviction_no, x);
}

uint64_t oracle_rand_key(uint64_t seed, int64_t eviction_no, int32_t x)
{
    uint64_t key = ((uint64_t)eviction_no << 32) + (uint64_t)(uint32_t)x;
    return splitmix64_mix(seed + 0x9E3779B97F4A7C15ull * key);
}

/* ============================================================ log replay ==
 *
 * Operator logs (Appendix C.6) lowered to storages, simulator tensors and
 * operators (Appendix C.1), and the eviction loop over storages:
 *   - CALL: an operator whose outputs are new tensors; an output described by
 *     ALIAS to nothing owns a new storage of its MEMORY size, one aliased to a
 *     name is a view (size 0) of that name's storage;
 *   - MUTATE: a pure operator whose outputs are clones (new storages of the
 *     same size) of the mutated inputs; the mutated names are rebound to the
 *     clones (Appendix C.6 "Supporting mutation");
 *   - CONSTANT: a nullary operator of cost 0 whose storage is pinned;
 *   - COPY, COPYFROM, RELEASE: external reference counts; a storage whose
 *     count drops to zero is released after the last operator issued;
 *   - tensors still referenced at the end are the required outputs.
 * A tensor is defined when its storage is resident and its operator ran after
 * the storage last became resident.  An operator call locks its inputs'
 * storages, defines undefined inputs in listed order (rematerialization),
 * allocates all its non-view outputs, runs, frees the new copies of outputs
 * that were already defined (Appendix C.4), and unlocks.  A storage's cost
 * sums, over every tensor that views it, the cost of that tensor's operator,
 * and its dependencies are the storages those operators read (Appendix C.2);
 * both cover the tensors that exist, so they grow when the first run of an
 * operator creates its tensors (the graph is indexed by time, and the cost
 * changes when a view is made); its staleness uses the latest reference to
 * any of its tensors.  Banishing a released storage needs every tensor computed from
 * it (outside it) defined or gone, and pins their resident storages.
 * Scoring, eviction, union-find, deallocation policies and search
 * approximations are the trace simulator's, run over storages.
 */

typedef struct {
    int32_t n_instrs, n_names;
    const int32_t *kind, *a, *b, *n_in;
    const int64_t *value, *list_offsets;
    const int32_t *ids;
} oracle_log;

enum { LG_MEMORY = 0, LG_ALIAS, LG_CALL, LG_MUTATE, LG_CONSTANT, LG_COPY, LG_COPYFROM, LG_RELEASE };

typedef struct { int64_t n, cap; int64_t *v; } vec64;
typedef struct { int64_t n, cap; int32_t *v; } vec32;

static int v64_push(vec64 *x, int64_t e)
{
    if (x->n == x->cap) {
        int64_t c = x->cap ? 2 * x->cap : 64;
        int64_t *p = realloc(x->v, sizeof(int64_t) * (size_t)c);
        if (!p) return -1;
        x->v = p;
        x->cap = c;
    }
    x->v[x->n++] = e;
    return 0;
}

static int v32_push(vec32 *x, int32_t e)
{
    if (x->n == x->cap) {
        int64_t c = x->cap ? 2 * x->cap : 64;
        int32_t *p = realloc(x->v, sizeof(int32_t) * (size_t)c);
        if (!p) return -1;
        x->v = p;
        x->cap = c;
    }
    x->v[x->n++] = e;
    return 0;
}

typedef struct {
    vec64 s_size, t_storage, t_op, t_alias, s_root, s_const, s_eref, t_eref;
    vec64 op_cost, in_off, out_off, rel_off;
    vec32 ins, outs, rel, req;
    int64_t F;
    /* storage-level metadata program: operator s produces storage s from its
     * parent storages, at the cost of the root's operator */
    oracle_trace meta;
    int64_t *m_size, *m_cost, *m_in_off;
    uint8_t *m_flags;
    int32_t *m_out, *m_in;
    int64_t *dt_off;              /* tensors computed from each storage (outside it) */
    int32_t *dt;
    graph g;
    int built;
} log_prog;

static void log_prog_free(log_prog *L)
{
    vec64 *v64s[] = {&L->s_size, &L->t_storage, &L->t_op, &L->t_alias, &L->s_root, &L->s_const, &L->s_eref,
                     &L->t_eref, &L->op_cost, &L->in_off, &L->out_off, &L->rel_off};
    for (size_t i = 0; i < sizeof(v64s) / sizeof(v64s[0]); i++) free(v64s[i]->v);
    free(L->ins.v); free(L->outs.v); free(L->rel.v); free(L->req.v);
    free(L->m_size); free(L->m_cost); free(L->m_in_off); free(L->m_flags); free(L->m_out); free(L->m_in);
    free(L->dt_off); free(L->dt);
    if (L->built) graph_free(&L->g);
    memset(L, 0, sizeof(*L));
}

/* external references: the storage released when its count reaches zero */
static int lg_ref(log_prog *L, int64_t t, int d)
{
    int64_t st = L->t_storage.v[t];
    L->t_eref.v[t] += d;
    L->s_eref.v[st] += d;
    if (L->t_eref.v[t] < 0 || L->s_eref.v[st] < 0) return -1;
    if (d < 0 && L->s_eref.v[st] == 0) {
        if (L->F == 0) return -1;
        if (v32_push(&L->rel, (int32_t)st)) return -1;
        L->rel_off.v[L->F]++;          /* counts per op, prefix-summed later */
    }
    return 0;
}

static int64_t lg_new_storage(log_prog *L, int64_t size, int constant, int64_t root)
{
    if (v64_push(&L->s_size, size) || v64_push(&L->s_const, constant) || v64_push(&L->s_root, root) ||
        v64_push(&L->s_eref, 0))
        return -1;
    return L->s_size.n - 1;
}

static int64_t lg_new_tensor(log_prog *L, int64_t storage, int64_t op, int alias)
{
    if (v64_push(&L->t_storage, storage) || v64_push(&L->t_op, op) || v64_push(&L->t_alias, alias) ||
        v64_push(&L->t_eref, 0))
        return -1;
    return L->t_storage.n - 1;
}

static int64_t lg_new_op(log_prog *L, int64_t cost)
{
    if (v64_push(&L->op_cost, cost) || v64_push(&L->rel_off, 0)) return -1;
    L->F++;
    return L->F - 1;
}

/* Lower a log; returns 0 or -2 on a malformed log. */
static int log_lower(log_prog *L, const oracle_log *lg)
{
    memset(L, 0, sizeof(*L));
    int32_t nn = lg->n_names > 0 ? lg->n_names : 1;
    int64_t *name = malloc(sizeof(int64_t) * (size_t)nn);     /* name -> tensor, -1 unbound */
    int64_t *local = malloc(sizeof(int64_t) * (size_t)nn);    /* names of one call's own storages */
    if (!name || !local) { free(name); free(local); return -1; }
    for (int32_t i = 0; i < nn; i++) name[i] = local[i] = -1;
    int rc = 0;
    if (v64_push(&L->rel_off, 0) || v64_push(&L->in_off, 0) || v64_push(&L->out_off, 0)) rc = -1;
#define BAD_NAME(x) ((x) < 0 || (x) >= lg->n_names)
    for (int32_t i = 0; i < lg->n_instrs && rc == 0;) {
        int32_t k = lg->kind[i];
        if (k == LG_CONSTANT) {
            int32_t nm = lg->a[i];
            if (i + 1 >= lg->n_instrs || lg->kind[i + 1] != LG_MEMORY || lg->a[i + 1] != nm || BAD_NAME(nm) ||
                name[nm] >= 0 || lg->value[i + 1] < 1) { rc = -2; break; }
            int64_t o = lg_new_op(L, 0);
            int64_t t = lg_new_tensor(L, -1, o, 0);
            int64_t st = lg_new_storage(L, lg->value[i + 1], 1, t);
            if (o < 0 || t < 0 || st < 0 || v32_push(&L->outs, (int32_t)t)) { rc = -1; break; }
            L->t_storage.v[t] = st;
            if (v64_push(&L->in_off, L->ins.n) || v64_push(&L->out_off, L->outs.n)) { rc = -1; break; }
            name[nm] = t;
            if (lg_ref(L, t, +1)) { rc = -2; break; }
            i += 2;
        } else if (k == LG_CALL || k == LG_MUTATE) {
            int64_t lo = lg->list_offsets[i], hi = lg->list_offsets[i + 1];
            int32_t nin = lg->n_in[i];
            int64_t nout = hi - lo - nin;
            if (nin < 0 || nout < 0 || lg->value[i] < 1 || (k == LG_CALL && nout < 1)) { rc = -2; break; }
            for (int64_t e = lo; e < lo + nin && rc == 0; e++) {
                int32_t nm = lg->ids[e];
                if (BAD_NAME(nm) || name[nm] < 0) rc = -2;
            }
            if (rc) break;
            int64_t o = lg_new_op(L, lg->value[i]);
            if (o < 0) { rc = -1; break; }
            for (int64_t e = lo; e < lo + nin; e++)
                if (v32_push(&L->ins, (int32_t)name[lg->ids[e]])) { rc = -1; break; }
            if (rc) break;
            if (k == LG_CALL) {
                if (i + 2 * nout >= lg->n_instrs) { rc = -2; break; }
                for (int64_t j = 0; j < nout && rc == 0; j++) {
                    int32_t nm = lg->ids[lo + nin + j];
                    int32_t mi = i + 1 + 2 * (int32_t)j, ai = mi + 1;
                    for (int64_t q = lo + nin; q < lo + nin + j; q++)
                        if (lg->ids[q] == nm) rc = -2;          /* an output name listed twice */
                    if (rc) break;
                    if (BAD_NAME(nm) || name[nm] >= 0 || local[nm] >= 0 || lg->kind[mi] != LG_MEMORY ||
                        lg->kind[ai] != LG_ALIAS || lg->a[mi] != nm || lg->a[ai] != nm) { rc = -2; break; }
                    int32_t src = lg->b[ai];
                    int64_t t;
                    if (src < 0) {
                        if (lg->value[mi] < 1) { rc = -2; break; }
                        t = lg_new_tensor(L, -1, o, 0);
                        int64_t st = lg_new_storage(L, lg->value[mi], 0, t);
                        if (t < 0 || st < 0) { rc = -1; break; }
                        L->t_storage.v[t] = st;
                        local[nm] = t;
                    } else {
                        /* a view of an input's storage or of one of this call's own new storages */
                        int64_t of = -1;
                        if (!BAD_NAME(src) && local[src] >= 0) of = local[src];
                        else if (!BAD_NAME(src) && name[src] >= 0) {
                            for (int64_t e = lo; e < lo + nin; e++)
                                if (lg->ids[e] == src) of = name[src];
                        }
                        if (of < 0) { rc = -2; break; }
                        t = lg_new_tensor(L, L->t_storage.v[of], o, 1);
                        if (t < 0) { rc = -1; break; }
                    }
                    if (v32_push(&L->outs, (int32_t)t)) { rc = -1; break; }
                }
                if (rc) break;
                for (int64_t j = 0; j < nout; j++) {
                    int32_t nm = lg->ids[lo + nin + j];
                    local[nm] = -1;
                    name[nm] = L->outs.v[L->outs.n - nout + j];
                    if (lg_ref(L, name[nm], +1)) { rc = -2; break; }
                }
                i += 1 + 2 * (int32_t)nout;
            } else {
                /* MUTATE: the mutated inputs (a subset of the inputs) become clones */
                int64_t first = L->outs.n;
                for (int64_t j = 0; j < nout && rc == 0; j++) {
                    int32_t nm = lg->ids[lo + nin + j];
                    int found = 0;
                    for (int64_t e = lo; e < lo + nin; e++) found |= lg->ids[e] == nm;
                    for (int64_t q = lo + nin; q < lo + nin + j; q++) found &= lg->ids[q] != nm;
                    if (!found) { rc = -2; break; }
                    int64_t old = name[nm];
                    int64_t t = lg_new_tensor(L, -1, o, 0);
                    int64_t st = lg_new_storage(L, L->s_size.v[L->t_storage.v[old]], 0, t);
                    if (t < 0 || st < 0 || v32_push(&L->outs, (int32_t)t)) { rc = -1; break; }
                    L->t_storage.v[t] = st;
                }
                if (rc) break;
                for (int64_t j = 0; j < nout && rc == 0; j++) {
                    int32_t nm = lg->ids[lo + nin + j];
                    int64_t old = name[nm];
                    name[nm] = L->outs.v[first + j];
                    if (lg_ref(L, name[nm], +1) || lg_ref(L, old, -1)) rc = -2;
                }
                i += 1;
            }
            if (rc == 0 && (v64_push(&L->in_off, L->ins.n) || v64_push(&L->out_off, L->outs.n))) rc = -1;
        } else if (k == LG_COPY) {
            int32_t to = lg->a[i], ti = lg->b[i];
            if (BAD_NAME(to) || BAD_NAME(ti) || name[to] >= 0 || name[ti] < 0) { rc = -2; break; }
            name[to] = name[ti];
            if (lg_ref(L, name[ti], +1)) rc = -2;
            i += 1;
        } else if (k == LG_COPYFROM) {
            int32_t to = lg->a[i], ti = lg->b[i];
            if (BAD_NAME(to) || BAD_NAME(ti) || name[to] < 0 || name[ti] < 0) { rc = -2; break; }
            int64_t old = name[to];
            name[to] = name[ti];
            if (lg_ref(L, name[ti], +1) || lg_ref(L, old, -1)) rc = -2;
            i += 1;
        } else if (k == LG_RELEASE) {
            int32_t nm = lg->a[i];
            if (BAD_NAME(nm) || name[nm] < 0) { rc = -2; break; }
            int64_t old = name[nm];
            name[nm] = -1;
            if (lg_ref(L, old, -1)) rc = -2;
            i += 1;
        } else {
            rc = -2;
        }
    }
#undef BAD_NAME
    free(name);
    free(local);
    if (rc) { log_prog_free(L); return rc; }
    /* release lists: counts per op -> offsets (events stay in log order) */
    for (int64_t o = 0; o < L->F; o++) L->rel_off.v[o + 1] += L->rel_off.v[o];
    for (int64_t t = 0; t < L->t_storage.n; t++)
        if (L->t_eref.v[t] > 0 && v32_push(&L->req, (int32_t)t)) { log_prog_free(L); return -1; }
    /* storage metadata program: tensors grouped by storage, then per storage
     * the distinct operators of its tensors, their cost and input storages */
    int64_t S = L->s_size.n, T = L->t_storage.n, F = L->F;
    size_t sn = (size_t)(S > 0 ? S : 1);
    int64_t *tb_off = calloc(sn + 1, sizeof(int64_t));
    int32_t *tb = malloc(sizeof(int32_t) * (size_t)(T > 0 ? T : 1));
    int64_t *seen_op = malloc(sizeof(int64_t) * (size_t)(F > 0 ? F : 1));
    int64_t *seen_st = malloc(sizeof(int64_t) * sn);
    L->m_size = malloc(sizeof(int64_t) * sn);
    L->m_cost = malloc(sizeof(int64_t) * sn);
    L->m_flags = calloc(sn, 1);
    L->m_out = malloc(sizeof(int32_t) * sn);
    L->m_in_off = calloc(sn + 1, sizeof(int64_t));
    L->dt_off = calloc(sn + 1, sizeof(int64_t));
    /* a storage's parents come from the operators of its tensors: at most
     * inputs x outputs over all operators */
    int64_t pbound = 1;
    for (int64_t o = 0; o < F; o++)
        pbound += (L->in_off.v[o + 1] - L->in_off.v[o]) * (L->out_off.v[o + 1] - L->out_off.v[o]);
    L->m_in = malloc(sizeof(int32_t) * (size_t)pbound);
    L->dt = malloc(sizeof(int32_t) * (size_t)pbound);
    if (!tb_off || !tb || !seen_op || !seen_st || !L->m_size || !L->m_cost || !L->m_flags || !L->m_out ||
        !L->m_in_off || !L->dt_off || !L->m_in || !L->dt) {
        free(tb_off); free(tb); free(seen_op); free(seen_st);
        log_prog_free(L);
        return -1;
    }
    for (int64_t t = 0; t < T; t++) tb_off[L->t_storage.v[t] + 1]++;
    for (int64_t st = 0; st < S; st++) tb_off[st + 1] += tb_off[st];
    {
        int64_t *fill = malloc(sizeof(int64_t) * sn);
        if (!fill) { free(tb_off); free(tb); free(seen_op); free(seen_st); log_prog_free(L); return -1; }
        for (int64_t st = 0; st < S; st++) fill[st] = tb_off[st];
        for (int64_t t = 0; t < T; t++) tb[fill[L->t_storage.v[t]]++] = (int32_t)t;
        free(fill);
    }
    for (int64_t o = 0; o < F; o++) seen_op[o] = -1;
    for (int64_t st = 0; st < S; st++) seen_st[st] = -1;
    int64_t w = 0;
    for (int64_t st = 0; st < S; st++) {
        L->m_size[st] = L->s_size.v[st];
        L->m_flags[st] = L->s_const.v[st] ? O_FLAG_CONSTANT : 0;
        L->m_out[st] = (int32_t)st;
        int64_t cost = 0;
        seen_st[st] = st;                       /* never its own parent */
        for (int64_t q = tb_off[st]; q < tb_off[st + 1]; q++) {
            int64_t o = L->t_op.v[tb[q]];
            cost += L->op_cost.v[o];           /* one term per tensor viewing the storage */
            if (seen_op[o] == st) continue;
            seen_op[o] = st;
            for (int64_t e = L->in_off.v[o]; e < L->in_off.v[o + 1]; e++) {
                int64_t p = L->t_storage.v[L->ins.v[e]];
                if (seen_st[p] == st) continue;
                seen_st[p] = st;
                L->m_in[w++] = (int32_t)p;
            }
        }
        L->m_cost[st] = L->s_const.v[st] ? 1 : cost;
        L->m_in_off[st + 1] = w;
    }
    free(tb_off); free(tb); free(seen_op); free(seen_st);
    /* tensors computed from each storage: outputs (of another storage) of
     * operators reading it; a pair repeats only within one operator, so the
     * operator's input storages are deduplicated first */
    {
        int64_t n_dt = 0;
        int64_t *cnt = calloc(sn + 1, sizeof(int64_t));
        int64_t *ps = malloc(sizeof(int64_t) * (size_t)pbound);
        int32_t *pt = malloc(sizeof(int32_t) * (size_t)pbound);
        int64_t *uniq = malloc(sizeof(int64_t) * (size_t)(L->ins.n > 0 ? L->ins.n : 1));
        if (!cnt || !ps || !pt || !uniq) { free(cnt); free(ps); free(pt); free(uniq); log_prog_free(L); return -1; }
        for (int64_t o = 0; o < F; o++) {
            int64_t nu = 0;
            for (int64_t e = L->in_off.v[o]; e < L->in_off.v[o + 1]; e++) {
                int64_t p = L->t_storage.v[L->ins.v[e]];
                int dup = 0;
                for (int64_t z = 0; z < nu && !dup; z++) dup = uniq[z] == p;
                if (!dup) uniq[nu++] = p;
            }
            for (int64_t z = 0; z < nu; z++)
                for (int64_t q = L->out_off.v[o]; q < L->out_off.v[o + 1]; q++) {
                    int32_t v = L->outs.v[q];
                    if (L->t_storage.v[v] == uniq[z]) continue;
                    ps[n_dt] = uniq[z];
                    pt[n_dt++] = v;
                    cnt[uniq[z] + 1]++;
                }
        }
        for (int64_t st = 0; st < S; st++) cnt[st + 1] += cnt[st];
        for (int64_t st = 0; st <= S; st++) L->dt_off[st] = cnt[st];
        for (int64_t z = 0; z < n_dt; z++) L->dt[cnt[ps[z]]++] = pt[z];
        free(cnt); free(ps); free(pt); free(uniq);
    }
    L->meta.n_tensors = (int32_t)S;
    L->meta.n_ops = (int32_t)S;
    L->meta.tensor_size = L->m_size;
    L->meta.tensor_flags = L->m_flags;
    L->meta.op_output = L->m_out;
    L->meta.op_cost = L->m_cost;
    L->meta.op_input_offsets = L->m_in_off;
    L->meta.op_inputs = L->m_in;
    if (graph_build(&L->g, &L->meta)) { log_prog_free(L); return -1; }
    L->built = 1;
    /* a constant storage has no parent operation and costs nothing */
    for (int64_t st = 0; st < S; st++)
        if (L->s_const.v[st]) { L->g.producer[st] = -1; L->g.c0[st] = 0; }
    return 0;
}

static int log_defined(const sim *s, const log_prog *L, int64_t t)
{
    int64_t st = L->t_storage.v[t];
    return s->state[st] == ST_RESIDENT && s->gen[t] == s->sgen[st];
}

/* Banishing over storages: st must be unheld, and every tensor computed from
 * it (outside it) defined or gone; the resident storages of those tensors are
 * pinned.  Otherwise st stays pending. */
static void log_try_banish(sim *s, int32_t st)
{
    const log_prog *L = s->logp;
    int blocked = s->locks[st] > 0;
    for (int64_t e = L->dt_off[st]; e < L->dt_off[st + 1] && !blocked; e++) {
        int32_t v = L->dt[e];
        blocked = !log_defined(s, L, v) && s->state[L->t_storage.v[v]] != ST_BANISHED;
    }
    if (blocked) { s->pending[st] = 1; return; }
    s->pending[st] = 0;
    if (s->state[st] == ST_RESIDENT) s->memory -= L->s_size.v[st];
    s->state[st] = ST_BANISHED;
    s->r[R_EAGER]++;
    for (int64_t e = L->dt_off[st]; e < L->dt_off[st + 1]; e++) {
        int64_t d = L->t_storage.v[L->dt[e]];
        if (s->state[d] == ST_RESIDENT) s->pinned[d] = 1;
    }
}

/* A replay's storage graph as of now (Appendix C.2, indexed by time): the
 * parents and children created so far and the cost of the tensors created so
 * far. */
static int64_t log_n_par(const sim *s, int32_t u) { return s->npar[u]; }
static int32_t log_par_at(const sim *s, int32_t u, int64_t k) { return s->dpar[u][k]; }
static int64_t log_n_ch(const sim *s, int32_t u) { return s->nch[u]; }
static int32_t log_ch_at(const sim *s, int32_t u, int64_t k) { return s->dch[u][k]; }
static int64_t log_c0_of(const sim *s, int32_t u) { return s->dc0[u]; }

static const graph_view LOG_VIEW = {log_n_par, log_par_at, log_n_ch, log_ch_at, log_c0_of, log_try_banish};

static int push32(int32_t **v, int64_t *n, int64_t *cap, int32_t e)
{
    if (*n == *cap) {
        int64_t c = *cap ? 2 * *cap : 4;
        int32_t *q = realloc(*v, sizeof(int32_t) * (size_t)c);
        if (!q) return -1;
        *v = q;
        *cap = c;
    }
    (*v)[(*n)++] = e;
    return 0;
}

/* The first run of operator o creates its tensors: each adds the operator's
 * cost to its storage's cost and makes the storages o reads (other than its
 * own) parents of it (Appendix C.2, over the tensors that exist). */
static void log_create(sim *s, const log_prog *L, int64_t o)
{
    for (int64_t q = L->out_off.v[o]; q < L->out_off.v[o + 1]; q++) {
        int32_t st = (int32_t)L->t_storage.v[L->outs.v[q]];
        if (!L->s_const.v[st]) s->dc0[st] += L->op_cost.v[o];
        for (int64_t e = L->in_off.v[o]; e < L->in_off.v[o + 1]; e++) {
            int32_t p = (int32_t)L->t_storage.v[L->ins.v[e]];
            if (p == st) continue;
            int known = 0;
            for (int64_t k = 0; k < s->npar[st] && !known; k++) known = s->dpar[st][k] == p;
            if (known) continue;
            if (push32(&s->dpar[st], &s->npar[st], &s->cpar[st], p) ||
                push32(&s->dch[p], &s->nch[p], &s->cch[p], st))
                abort();
        }
    }
}

/* run operator o (a rematerialization if remat), defining its outputs */
static void log_call(sim *s, const log_prog *L, int64_t o, int remat)
{
    const int64_t ib = L->in_off.v[o], ie = L->in_off.v[o + 1];
    const int64_t ob = L->out_off.v[o], oe = L->out_off.v[o + 1];
    for (int64_t e = ib; e < ie; e++) lock(s, (int32_t)L->t_storage.v[L->ins.v[e]]);
    for (int64_t e = ib; e < ie; e++) {
        int32_t u = L->ins.v[e];
        if (!log_defined(s, L, u)) {
            log_call(s, L, L->t_op.v[u], 1);
            if (s->stopped) return;
        }
    }
    int64_t need = 0;
    for (int64_t e = ob; e < oe; e++)
        if (!L->t_alias.v[L->outs.v[e]]) need += L->s_size.v[L->t_storage.v[L->outs.v[e]]];
    allocate(s, need);
    if (s->stopped) return;
    for (int64_t e = ib; e < ie; e++) s->last_access[L->t_storage.v[L->ins.v[e]]] = s->clock;
    for (int64_t e = ob; e < oe; e++) s->last_access[L->t_storage.v[L->outs.v[e]]] = s->clock;
    int64_t c = L->op_cost.v[o];
    s->clock += c;
    s->r[R_TOTAL_COST] += c;
    s->r[R_EXECUTED]++;
    if (remat) { s->r[R_REMATS]++; s->r[R_REMAT_COST] += c; }
    else s->r[R_BASE_COST] += c;
    s->memory += need;
    if (s->memory > s->peak) s->peak = s->memory;
    for (int64_t e = ob; e < oe; e++) {
        int32_t v = L->outs.v[e];
        if (L->t_alias.v[v]) continue;
        int32_t st = (int32_t)L->t_storage.v[v];
        if (s->state[st] == ST_RESIDENT) { s->memory -= L->s_size.v[st]; continue; }   /* copy of a defined output */
        int was_evicted = s->state[st] == ST_EVICTED;
        s->state[st] = ST_RESIDENT;
        s->gen[v] = ++s->sgen[st];
        if (uses_uf(s->heuristic)) {
            if (was_evicted) {
                int32_t r = uf_find(s, s->node_of[st]);
                s->uf_cost[r] -= c0_of(s, st);
            }
            int32_t nd = uf_new(s);
            if (nd < 0) abort();
            s->node_of[st] = nd;
        }
    }
    for (int64_t e = ob; e < oe; e++) {
        int32_t v = L->outs.v[e];
        if (L->t_alias.v[v]) s->gen[v] = s->sgen[L->t_storage.v[v]];
    }
    if (!remat) log_create(s, L, o);
    if (s->clock >= CLOCK_LIMIT) { s->r[R_STATUS] = OS_CLOCK_OVERFLOW; s->stopped = OS_CLOCK_OVERFLOW; return; }
    for (int64_t e = ib; e < ie; e++) unlock(s, (int32_t)L->t_storage.v[L->ins.v[e]]);
    if (remat && s->policy == OP_BANISH)
        for (int64_t e = ib; e < ie; e++) {
            int32_t st = (int32_t)L->t_storage.v[L->ins.v[e]];
            if (s->pending[st]) try_banish(s, st);
        }
}

static void log_run(sim *s, const log_prog *L)
{
    s->r[R_FAILED_OP] = -1;
    for (int64_t o = 0; o < L->F; o++) {
        s->cur_op = o;
        log_call(s, L, o, 0);
        if (s->stopped) goto done;
        for (int64_t e = L->rel_off.v[o]; e < L->rel_off.v[o + 1]; e++) release(s, L->rel.v[e]);
    }
    s->cur_op = L->F;
    for (int64_t k = 0; k < L->req.n; k++) {
        int32_t t = L->req.v[k];
        lock(s, (int32_t)L->t_storage.v[t]);
        if (!log_defined(s, L, t)) {
            log_call(s, L, L->t_op.v[t], 1);
            if (s->stopped) goto done;
        }
    }
done:
    if (s->stopped == OS_OOM || s->stopped == OS_CLOCK_OVERFLOW) s->r[R_FAILED_OP] = s->cur_op;
    s->r[R_PEAK] = s->peak;
    s->r[R_FINAL_MEM] = s->memory;
}

static int run_one_log(const log_prog *L, const oracle_spec *sp, int64_t *result)
{
    int64_t S = L->s_size.n, T = L->t_storage.n;
    sim s;
    memset(&s, 0, sizeof(s));
    s.g = &L->g;
    s.view = &LOG_VIEW;
    s.tr = &L->meta;
    s.logp = L;
    s.heuristic = sp->heuristic;
    s.policy = sp->policy;
    s.search = sp->search;
    s.budget = sp->budget;
    s.seed = sp->seed;
    size_t sn = (size_t)(S > 0 ? S : 1), tn = (size_t)(T > 0 ? T : 1);
    s.state = calloc(sn, 1);
    s.pinned = calloc(sn, 1);
    s.pending = calloc(sn, 1);
    s.locks = calloc(sn, sizeof(int32_t));
    s.last_access = calloc(sn, sizeof(int64_t));
    s.node_of = malloc(sizeof(int32_t) * sn);
    s.queue = malloc(sizeof(int32_t) * sn);
    s.mark = calloc(sn, sizeof(int64_t));
    s.sgen = calloc(sn, sizeof(int64_t));
    s.gen = malloc(sizeof(int64_t) * tn);
    s.dc0 = calloc(sn, sizeof(int64_t));
    s.dpar = calloc(sn, sizeof(int32_t *));
    s.dch = calloc(sn, sizeof(int32_t *));
    s.npar = calloc(sn, sizeof(int64_t));
    s.nch = calloc(sn, sizeof(int64_t));
    s.cpar = calloc(sn, sizeof(int64_t));
    s.cch = calloc(sn, sizeof(int64_t));
    int rc = 0;
    if (!s.state || !s.pinned || !s.pending || !s.locks || !s.last_access || !s.node_of || !s.queue || !s.mark ||
        !s.sgen || !s.gen || !s.dc0 || !s.dpar || !s.dch || !s.npar || !s.nch || !s.cpar || !s.cch)
        rc = -1;
    else {
        for (int64_t i = 0; i < S; i++) s.node_of[i] = -1;
        for (int64_t i = 0; i < T; i++) s.gen[i] = -1;
        for (int64_t i = 0; i < S; i++) s.pinned[i] = (uint8_t)L->s_const.v[i];
        log_run(&s, L);
        for (int i = 0; i < R_NFIELDS; i++) result[i] = s.r[i];
    }
    free(s.state); free(s.pinned); free(s.pending); free(s.locks); free(s.last_access); free(s.node_of);
    free(s.queue); free(s.mark); free(s.sgen); free(s.gen);
    for (int64_t i = 0; i < S && s.dpar && s.dch; i++) { free(s.dpar[i]); free(s.dch[i]); }
    free(s.dc0); free(s.dpar); free(s.dch); free(s.npar); free(s.nch); free(s.cpar); free(s.cch);
    free(s.uf_parent); free(s.uf_cost); free(s.uf_mark);
    return rc;
}

typedef struct {
    const log_prog *progs;
    const oracle_spec *specs;
    int64_t *results;
    int32_t n_sims, next;
    pthread_mutex_t mu;
    int rc;
} log_batch;

static void *log_worker(void *arg)
{
    log_batch *b = arg;
    for (;;) {
        pthread_mutex_lock(&b->mu);
        int32_t i = b->next++;
        pthread_mutex_unlock(&b->mu);
        if (i >= b->n_sims) break;
        int rc = run_one_log(&b->progs[b->specs[i].trace], &b->specs[i], b->results + (int64_t)i * R_NFIELDS);
        if (rc) { pthread_mutex_lock(&b->mu); b->rc = rc; pthread_mutex_unlock(&b->mu); }
    }
    return NULL;
}

/* Replay n_sims simulations over n_logs operator logs on n_threads threads.
 * Returns 0, -1 on allocation failure, -2 on a bad argument or a malformed
 * log. */
int oracle_run_log(const oracle_log *logs, int32_t n_logs, const oracle_spec *specs, int32_t n_sims,
                   int64_t *results, int32_t n_threads)
{
    if (n_logs < 0 || n_sims < 0) return -2;
    for (int32_t i = 0; i < n_sims; i++)
        if (specs[i].trace < 0 || specs[i].trace >= n_logs ||
            !((specs[i].heuristic >= 0 && specs[i].heuristic <= OH_MSPS) || family(specs[i].heuristic)) ||
            specs[i].policy < OP_EAGER || specs[i].policy > OP_BANISH ||
            specs[i].search < 0 || specs[i].search > (OSR_IGNORE_SMALL | OSR_SAMPLE) ||
            (specs[i].policy == OP_BANISH && uses_uf(specs[i].heuristic)))
            return -2;
    log_prog *progs = calloc((size_t)(n_logs > 0 ? n_logs : 1), sizeof(log_prog));
    if (!progs) return -1;
    int rc = 0;
    int32_t built = 0;
    for (; built < n_logs; built++)
        if ((rc = log_lower(&progs[built], &logs[built])) != 0) break;
    if (rc == 0) {
        log_batch b;
        memset(&b, 0, sizeof(b));
        b.progs = progs; b.specs = specs; b.results = results; b.n_sims = n_sims;
        pthread_mutex_init(&b.mu, NULL);
        if (n_threads < 1) n_threads = 1;
        if (n_threads > n_sims) n_threads = n_sims > 0 ? n_sims : 1;
        pthread_t *th = calloc((size_t)n_threads, sizeof(pthread_t));
        pthread_attr_t attr;
        pthread_attr_init(&attr);
        pthread_attr_setstacksize(&attr, WORKER_STACK);
        int started = 0;
        if (th)
            for (; started < n_threads; started++)
                if (pthread_create(&th[started], &attr, log_worker, &b)) break;
        if (started == 0) log_worker(&b);
        for (int k = 0; k < started; k++) pthread_join(th[k], NULL);
        pthread_attr_destroy(&attr);
        free(th);
        pthread_mutex_destroy(&b.mu);
        rc = b.rc;
    }
    for (int32_t i = 0; i < built; i++) log_prog_free(&progs[i]);
    free(progs);
    return rc;
}
