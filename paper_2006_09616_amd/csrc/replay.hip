// replay.hip -- gfx950 kernels of the batched DTR eviction-loop simulator.
//
// One wavefront (64 lanes, one workgroup) owns one simulation at a time and
// pulls the next one from a global work counter (persistent grid).  The
// sequential part of DTR's operator call (Section 2; Appendix C.4) runs
// wave-uniformly: every lane holds the same clock, memory and counters.  The
// data-parallel part -- scoring every evictable tensor when memory runs out
// (Appendix C.4 "Runtime state": the lowest score is evicted) -- is spread
// over the lanes: each lane scores a strided slice of the pool, keeps its own
// lexicographic (score, id) minimum, and a cross-lane reduction yields the
// victim.  Scores N/D are compared exactly by 128-bit cross-multiplication.
//
// Neighbourhood costs:
//   h_DTR^eq  union-find over evicted components with a running cost per set;
//             a tensor's new node is created when it is evicted and unioned
//             with its evicted neighbours' sets; rematerialization subtracts
//             c0 from the set and detaches the tensor (split approximation,
//             Appendix C.2).  A query sums the distinct sets of the evicted
//             parents and children without merging them.
//   h_DTR     e* (Appendix C.2): each lane walks evicted ancestors and
//             evicted descendants of its candidate with lane-private epoch
//             stamps (set semantics, nothing counted twice).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout.h"

namespace dtr {

typedef unsigned __int128 u128;

enum { H_DTR = 0, H_EQ = 1, H_LOCAL = 2, H_LRU = 3, H_SIZE = 4, H_RAND = 5, H_ESTAR = 6 };
enum { ST_OK = 0, ST_OOM = 1, ST_CLOCK = 2, ST_CAPACITY = 3 };

constexpr uint8_t FLAG_CONST = 1;

__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ int64_t uni64(int64_t v)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014)
__device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// a strictly better (lower score) than b; ties go to the smaller id
__device__ __forceinline__ bool better(uint64_t na, u128 da, int32_t ia, uint64_t nb, u128 db, int32_t ib)
{
    u128 l = (u128)na * db;
    u128 r = (u128)nb * da;
    if (l != r) return l < r;
    return ia < ib;
}

struct Slot {
    int32_t *sw, *locks, *pos;
    int64_t *last;
    int32_t *pool_id;
    int64_t *pool_last, *pool_size, *pool_c0;
    int32_t *stack;
    int32_t *uf_parent, *uf_size, *uf_remap;
    int64_t *uf_cost;
    uint32_t *stamp;
    int32_t *queue;
    int64_t uf_cap;
    int32_t n_max;
};

__device__ __forceinline__ Slot slot_at(const KernelArgs &a, int32_t k)
{
    uint8_t *b = a.slots + (size_t)k * (size_t)a.L.bytes;
    Slot S;
    S.sw = (int32_t *)(b + a.L.sw);
    S.locks = (int32_t *)(b + a.L.locks);
    S.last = (int64_t *)(b + a.L.last);
    S.pos = (int32_t *)(b + a.L.pos);
    S.pool_id = (int32_t *)(b + a.L.pool_id);
    S.pool_last = (int64_t *)(b + a.L.pool_last);
    S.pool_size = (int64_t *)(b + a.L.pool_size);
    S.pool_c0 = (int64_t *)(b + a.L.pool_c0);
    S.stack = (int32_t *)(b + a.L.stack);
    S.uf_parent = (int32_t *)(b + a.L.uf_parent);
    S.uf_cost = (int64_t *)(b + a.L.uf_cost);
    S.uf_size = (int32_t *)(b + a.L.uf_size);
    S.uf_remap = (int32_t *)(b + a.L.uf_remap);
    S.stamp = (uint32_t *)(b + a.L.stamp);
    S.queue = (int32_t *)(b + a.L.queue);
    S.uf_cap = a.L.uf_cap;
    S.n_max = (int32_t)a.L.n_max;
    return S;
}

// Wave-uniform simulation state.
struct Sim {
    TraceDev t;
    Slot S;
    int32_t h;
    int32_t lane;
    int64_t budget;
    uint64_t seed;
    int64_t T, mem, peak;
    int32_t pool_n;
    int32_t uf_n;
    int32_t status, cur_op;
    uint32_t epoch;
    int64_t evict_no;
    int64_t total, base, remat_cost, executed, remats, evictions, eager, scores;
    int64_t nbr, adj;     // per-lane partial sums, reduced at the end
};

// ---------------------------------------------------------------- pool ----

__device__ __forceinline__ void pool_add(Sim &s, int32_t x)
{
    if (s.pool_n >= s.S.n_max) { s.status = ST_CAPACITY; return; }   // a tensor joins at most once
    int32_t i = s.pool_n++;
    s.S.pool_id[i] = x;
    s.S.pool_last[i] = s.S.last[x];
    s.S.pool_size[i] = s.t.size[x];
    s.S.pool_c0[i] = s.t.c0[x];
    s.S.pos[x] = i;
}

__device__ __forceinline__ void pool_remove(Sim &s, int32_t x)
{
    int32_t i = uni(s.S.pos[x]);
    int32_t j = --s.pool_n;
    if (i != j) {
        int32_t y = uni(s.S.pool_id[j]);
        int64_t l = s.S.pool_last[j], z = s.S.pool_size[j], c = s.S.pool_c0[j];
        s.S.pool_id[i] = y;
        s.S.pool_last[i] = l;
        s.S.pool_size[i] = z;
        s.S.pool_c0[i] = c;
        s.S.pos[y] = i;
    }
}

__device__ __forceinline__ bool evictable_resident(const Sim &s, int32_t x)
{
    return s.S.sw[x] == SW_RESIDENT && s.S.locks[x] == 0 && !(s.t.flags[x] & FLAG_CONST);
}

__device__ __forceinline__ void lock(Sim &s, int32_t u)
{
    int32_t l = uni(s.S.locks[u]) + 1;
    s.S.locks[u] = l;
    if (l == 1 && uni(s.S.sw[u]) == SW_RESIDENT && !(s.t.flags[u] & FLAG_CONST)) pool_remove(s, u);
}

__device__ __forceinline__ void unlock(Sim &s, int32_t u)
{
    int32_t l = uni(s.S.locks[u]) - 1;
    s.S.locks[u] = l;
    if (l == 0 && uni(s.S.sw[u]) == SW_RESIDENT && !(s.t.flags[u] & FLAG_CONST)) pool_add(s, u);
}

// ---------------------------------------------------------- union-find ----

__device__ __forceinline__ int32_t find_ro(const int32_t *parent, int32_t x, int32_t limit)
{
    for (int32_t k = 0; k <= limit; k++) {
        int32_t p = parent[x];
        if (p == x) return x;
        x = p;
    }
    return -1;   // not a forest: reported as a capacity error
}

__device__ __forceinline__ int32_t find_compress(Sim &s, int32_t x)
{
    int32_t *P = s.S.uf_parent;
    int32_t root = x;
    for (int32_t k = 0;; k++) {
        int32_t p = uni(P[root]);
        if (p == root) break;
        if (k > s.uf_n) { s.status = ST_CAPACITY; return x; }
        root = p;
    }
    while (x != root) {
        int32_t nx = uni(P[x]);
        P[x] = root;
        x = nx;
    }
    return root;
}

// Rebuild the node pool: one node per distinct set that still holds an
// evicted tensor (sets left with phantom members only are unreachable).
// Membership and running costs are unchanged, so every later query is too.
__device__ __forceinline__ void uf_compact(Sim &s)
{
    const int32_t lane = s.lane, n = s.t.n;
    int32_t *P = s.S.uf_parent, *R = s.S.uf_remap, *sw = s.S.sw, *tmp = s.S.pos;
    for (int32_t i = lane; i < s.uf_n; i += WAVE) R[i] = -1;
    __syncthreads();
    for (int32_t x = lane; x < n; x += WAVE) {
        int32_t v = sw[x];
        if (v >= 0) {
            int32_t r = find_ro(P, v, s.uf_n);
            if (r < 0) r = v;    // cannot happen in a forest; keeps indices in range
            tmp[x] = r;          // pos[] is unused while a tensor is evicted
            R[r] = 0;
        }
    }
    __syncthreads();
    int32_t kept = 0;
    for (int32_t base = 0; base < s.uf_n; base += WAVE) {
        int32_t i = base + lane;
        bool keep = i < s.uf_n && R[i] == 0;
        int64_t c = keep ? s.S.uf_cost[i] : 0;
        uint64_t m = __ballot(keep);
        int32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
        __syncthreads();
        if (keep) {
            int32_t ni = kept + rank;
            R[i] = ni;
            s.S.uf_cost[ni] = c;
            P[ni] = ni;
            s.S.uf_size[ni] = 1;
        }
        kept += __popcll(m);
        __syncthreads();
    }
    for (int32_t x = lane; x < n; x += WAVE) {
        if (sw[x] >= 0) sw[x] = R[tmp[x]];
    }
    __syncthreads();
    s.uf_n = kept;
}

__device__ __forceinline__ int32_t unite(Sim &s, int32_t a, int32_t b)
{
    if (a == b) return a;
    int32_t sa = uni(s.S.uf_size[a]), sb = uni(s.S.uf_size[b]);
    if (sa < sb) { int32_t t = a; a = b; b = t; }
    int64_t cb = uni64(s.S.uf_cost[b]);
    int64_t ca = uni64(s.S.uf_cost[a]);
    s.S.uf_parent[b] = a;
    s.S.uf_size[a] = sa + sb;
    s.S.uf_cost[a] = ca + cb;
    return a;
}

// ------------------------------------------------------------ eviction ----

__device__ __forceinline__ bool evict(Sim &s, int32_t v, bool eager)
{
    if (s.h == H_EQ) {
        if (s.uf_n >= s.S.uf_cap) {
            uf_compact(s);
            if (s.uf_n >= s.S.uf_cap) { s.status = ST_CAPACITY; return false; }
        }
        int32_t nd = s.uf_n++;
        s.S.uf_parent[nd] = nd;
        s.S.uf_size[nd] = 1;
        s.S.uf_cost[nd] = s.t.c0[v];
        int32_t r = nd;
        const int32_t b = s.t.adj_off[v], e = s.t.adj_off[v + 1];
        for (int32_t k = b; k < e; k++) {
            int32_t w = s.t.adj[k];
            int32_t q = uni(s.S.sw[w]);
            if (q >= 0) r = unite(s, r, find_compress(s, q));
        }
        s.S.sw[v] = nd;
    } else {
        s.S.sw[v] = 0;
    }
    s.mem -= s.t.size[v];
    pool_remove(s, v);
    if (eager) s.eager++;
    else s.evictions++;
    return true;
}

// ---------------------------------------------------------------- scan ----

// Neighbourhood cost of candidate x under h_DTR^eq: distinct sets of the
// evicted parents and children.  The last eight distinct roots are kept in
// registers; past eight the earlier neighbours are re-checked.
__device__ __forceinline__ int64_t eq_cost(const Sim &s, int32_t x, int64_t &ev_count, bool &bad)
{
    const int32_t b = s.t.adj_off[x], e = s.t.adj_off[x + 1];
    const int32_t *P = s.S.uf_parent;
    int32_t r0 = -1, r1 = -1, r2 = -1, r3 = -1, r4 = -1, r5 = -1, r6 = -1, r7 = -1;
    int32_t distinct = 0;
    int64_t sum = 0, cnt = 0;
    for (int32_t k = b; k < e; k++) {
        int32_t w = s.t.adj[k];
        int32_t q = s.S.sw[w];
        if (q < 0) continue;
        cnt++;
        int32_t r = find_ro(P, q, s.uf_n);
        if (r < 0) { bad = true; break; }
        bool dup = (r == r0) | (r == r1) | (r == r2) | (r == r3) | (r == r4) | (r == r5) | (r == r6) | (r == r7);
        if (!dup && distinct > 8) {
            for (int32_t j = b; j < k && !dup; j++) {
                int32_t q2 = s.S.sw[s.t.adj[j]];
                if (q2 >= 0 && find_ro(P, q2, s.uf_n) == r) dup = true;
            }
        }
        if (!dup) {
            sum += s.S.uf_cost[r];
            r7 = r6; r6 = r5; r5 = r4; r4 = r3; r3 = r2; r2 = r1; r1 = r0; r0 = r;
            distinct++;
        }
    }
    ev_count = cnt;
    return sum;
}

// e*(x): evicted ancestors through evicted parents, then evicted descendants
// through evicted children; lane-private stamps make it a set.
__device__ __forceinline__ int64_t estar_cost(const Sim &s, int32_t x, uint32_t ep, int64_t &count)
{
    const int32_t lane = s.lane;
    uint32_t *st = s.S.stamp;
    int32_t *q = s.S.queue;
    int64_t sum = 0, cnt = 0;
    int32_t head = 0, tail = 0;
    q[(size_t)tail++ * WAVE + lane] = x;
    while (head < tail) {
        int32_t u = q[(size_t)head++ * WAVE + lane];
        int32_t o = s.t.producer[u];
        if (o < 0) continue;
        for (int32_t k = s.t.in_off[o], e = s.t.in_off[o + 1]; k < e; k++) {
            int32_t p = s.t.in[k];
            if (s.S.sw[p] < 0) continue;
            size_t sp = (size_t)p * WAVE + lane;
            if (st[sp] == ep) continue;
            st[sp] = ep;
            sum += s.t.c0[p];
            cnt++;
            q[(size_t)tail++ * WAVE + lane] = p;
        }
    }
    head = tail = 0;
    q[(size_t)tail++ * WAVE + lane] = x;
    while (head < tail) {
        int32_t u = q[(size_t)head++ * WAVE + lane];
        for (int32_t k = s.t.ch_off[u], e = s.t.ch_off[u + 1]; k < e; k++) {
            int32_t c = s.t.ch[k];
            if (s.S.sw[c] < 0) continue;
            size_t sc = (size_t)c * WAVE + lane;
            if (st[sc] == ep) continue;
            st[sc] = ep;
            sum += s.t.c0[c];
            cnt++;
            q[(size_t)tail++ * WAVE + lane] = c;
        }
    }
    count = cnt;
    return sum;
}

__device__ __forceinline__ void clear_stamps(Sim &s)
{
    for (size_t i = s.lane; i < (size_t)s.t.n * WAVE; i += WAVE) s.S.stamp[i] = 0;
    __syncthreads();
    s.epoch = 0;
}

// Score every pool entry; return the victim (uniform), or -1 if the pool is empty.
__device__ __forceinline__ int32_t scan(Sim &s)
{
    const int32_t n_pool = s.pool_n;
    const int32_t lane = s.lane;
    const int64_t T = s.T;
    bool have = false, bad = false;
    uint64_t bN = 0;
    u128 bD = 1;
    int32_t bid = 0x7fffffff;
    if ((s.h == H_DTR || s.h == H_ESTAR) &&
        (uint64_t)s.epoch + (uint64_t)(n_pool / WAVE) + 2 >= 0xffffffffull)
        clear_stamps(s);
    for (int32_t i0 = 0; i0 < n_pool; i0 += WAVE) {
        const int32_t i = i0 + lane;
        const uint32_t ep = ++s.epoch;   // uniform; one walk per lane per round
        if (i >= n_pool) continue;
        const int32_t x = s.S.pool_id[i];
        uint64_t N;
        u128 D;
        switch (s.h) {
        case H_LRU: {
            N = 1;
            D = (u128)(uint64_t)(T - s.S.pool_last[i]);
            break;
        }
        case H_SIZE: {
            N = 1;
            D = (u128)(uint64_t)s.S.pool_size[i];
            break;
        }
        case H_RAND: {
            uint64_t key = ((uint64_t)s.evict_no << 32) + (uint64_t)(uint32_t)x;
            N = mix64(s.seed + 0x9E3779B97F4A7C15ull * key);
            D = 1;
            break;
        }
        case H_LOCAL: {
            N = (uint64_t)s.S.pool_c0[i];
            D = (u128)(uint64_t)s.S.pool_size[i] * (u128)(uint64_t)(T - s.S.pool_last[i]);
            break;
        }
        case H_EQ: {
            int64_t ev;
            N = (uint64_t)(s.S.pool_c0[i] + eq_cost(s, x, ev, bad));
            D = (u128)(uint64_t)s.S.pool_size[i] * (u128)(uint64_t)(T - s.S.pool_last[i]);
            s.nbr += ev;
            s.adj += s.t.adj_off[x + 1] - s.t.adj_off[x];
            break;
        }
        default: {   // H_DTR, H_ESTAR
            int64_t cnt;
            N = (uint64_t)(s.S.pool_c0[i] + estar_cost(s, x, ep, cnt));
            if (s.h == H_DTR)
                D = (u128)(uint64_t)s.S.pool_size[i] * (u128)(uint64_t)(T - s.S.pool_last[i]);
            else
                D = (u128)(uint64_t)s.S.pool_size[i];
            s.nbr += cnt;
            s.adj += s.t.adj_off[x + 1] - s.t.adj_off[x];
            break;
        }
        }
        if (!have || better(N, D, x, bN, bD, bid)) {
            have = true;
            bN = N;
            bD = D;
            bid = x;
        }
    }
    // cross-lane lexicographic minimum
    int32_t hv = have ? 1 : 0;
    for (int off = WAVE / 2; off >= 1; off >>= 1) {
        uint64_t oN = __shfl_xor(bN, off, WAVE);
        uint64_t oDl = __shfl_xor((uint64_t)bD, off, WAVE);
        uint64_t oDh = __shfl_xor((uint64_t)(bD >> 64), off, WAVE);
        int32_t oid = __shfl_xor(bid, off, WAVE);
        int32_t oh = __shfl_xor(hv, off, WAVE);
        u128 oD = ((u128)oDh << 64) | oDl;
        if (oh && (!hv || better(oN, oD, oid, bN, bD, bid))) {
            hv = 1;
            bN = oN;
            bD = oD;
            bid = oid;
        }
    }
    if (__ballot(bad)) { s.status = ST_CAPACITY; return -1; }
    return uni(hv) ? uni(bid) : -1;
}

// ----------------------------------------------------- operator calls ----

__device__ __forceinline__ bool allocate(Sim &s, int64_t sz)
{
    while (s.mem + sz > s.budget) {
        if (s.pool_n == 0) { s.status = ST_OOM; return false; }
        int32_t v = scan(s);
        if (s.status != ST_OK) return false;
        s.scores += s.pool_n;
        if (!evict(s, v, false)) return false;
        s.evict_no++;
    }
    return true;
}

__device__ __forceinline__ bool execute(Sim &s, int32_t o, int32_t t, bool remat)
{
    const int32_t b = s.t.in_off[o], e = s.t.in_off[o + 1];
    for (int32_t k = b; k < e; k++) s.S.last[s.t.in[k]] = s.T;
    s.S.last[t] = s.T;
    const int64_t c = s.t.cost[o];
    s.T += c;
    s.total += c;
    s.executed++;
    if (remat) { s.remats++; s.remat_cost += c; }
    else s.base += c;
    s.mem += s.t.size[t];
    if (s.mem > s.peak) s.peak = s.mem;
    if (s.h == H_EQ && remat) {
        int32_t r = find_compress(s, uni(s.S.sw[t]));
        s.S.uf_cost[r] = uni64(s.S.uf_cost[r]) - s.t.c0[t];
    }
    s.S.sw[t] = SW_RESIDENT;
    if (s.T >= CLOCK_LIMIT) { s.status = ST_CLOCK; return false; }
    return true;
}

// Run the operation producing `root` together with every rematerialization it
// needs (explicit stack instead of recursion).  root_remat: the root itself is
// a rematerialization (output condition).  Returns false once the simulation
// has stopped.
__device__ __forceinline__ bool call(Sim &s, int32_t root, bool root_remat)
{
    int32_t sp = 0;
    int32_t tt = root, cur = -1;
    bool remat = root_remat;
    for (;;) {
        const int32_t o = uni(s.t.producer[tt]);
        const int32_t b = uni(s.t.in_off[o]), e = uni(s.t.in_off[o + 1]);
        if (cur < 0) {
            for (int32_t k = b; k < e; k++) lock(s, uni(s.t.in[k]));
            cur = 0;
        }
        if (cur < e - b) {
            const int32_t u = uni(s.t.in[b + cur]);
            cur++;
            if (uni(s.S.sw[u]) >= 0) {
                if (sp + 1 >= s.S.n_max) { s.status = ST_CAPACITY; return false; }
                s.S.stack[2 * sp] = tt;
                s.S.stack[2 * sp + 1] = cur;
                sp++;
                tt = u;
                cur = -1;
                remat = true;
            }
            continue;
        }
        if (s.status != ST_OK || !allocate(s, s.t.size[tt])) return false;
        if (!execute(s, o, tt, remat)) return false;
        for (int32_t k = b; k < e; k++) unlock(s, uni(s.t.in[k]));
        if (uni(s.S.locks[tt]) == 0) pool_add(s, tt);
        if (sp == 0) return true;
        sp--;
        tt = uni(s.S.stack[2 * sp]);
        cur = uni(s.S.stack[2 * sp + 1]);
        remat = sp > 0 ? true : root_remat;
    }
}

__device__ __forceinline__ void run_sim(const KernelArgs &a, int32_t sim, const Slot &S, int32_t lane)
{
    Sim s;
    const SpecDev sp = a.specs[sim];
    s.t = a.traces[sp.trace];
    s.S = S;
    s.h = sp.heuristic;
    s.lane = lane;
    s.budget = sp.budget;
    s.seed = sp.seed;
    s.T = 0;
    s.pool_n = 0;
    s.uf_n = 0;
    s.status = ST_OK;
    s.cur_op = 0;
    s.epoch = 0;
    s.evict_no = 0;
    s.total = s.base = s.remat_cost = s.executed = s.remats = s.evictions = s.eager = s.scores = 0;
    s.nbr = s.adj = 0;

    const int32_t n = s.t.n;
    for (int32_t x = lane; x < n; x += WAVE) {
        s.S.sw[x] = (s.t.flags[x] & FLAG_CONST) ? SW_RESIDENT : SW_UNCOMPUTED;
        s.S.locks[x] = 0;
        s.S.last[x] = 0;
    }
    if (s.h == H_DTR || s.h == H_ESTAR) clear_stamps(s);
    __syncthreads();
    s.mem = s.t.const_mem;
    s.peak = s.mem;

    bool ok = true;
    if (s.mem > s.budget) { s.status = ST_OOM; ok = false; }
    for (int32_t o = 0; ok && o < s.t.F; o++) {
        s.cur_op = o;
        if (!call(s, uni(s.t.out[o]), false) || s.status != ST_OK) { ok = false; break; }
        for (int32_t k = uni(s.t.rel_off[o]), e = uni(s.t.rel_off[o + 1]); ok && k < e; k++) {
            const int32_t r = uni(s.t.rel[k]);
            if (evictable_resident(s, r) && !evict(s, r, true)) ok = false;
        }
        if (s.status != ST_OK) ok = false;
    }
    if (ok) {
        s.cur_op = s.t.F;
        for (int32_t k = 0; k < s.t.n_req; k++) {
            const int32_t r = uni(s.t.req[k]);
            lock(s, r);
            if (uni(s.S.sw[r]) >= 0 && !call(s, r, true)) { ok = false; break; }
        }
    }

    int64_t nbr = s.nbr, adj = s.adj;
    for (int off = WAVE / 2; off >= 1; off >>= 1) {
        nbr += __shfl_xor(nbr, off, WAVE);
        adj += __shfl_xor(adj, off, WAVE);
    }
    if (lane == 0) {
        ResultDev r;
        r.total_cost = s.total;
        r.base_cost = s.base;
        r.remat_cost = s.remat_cost;
        r.peak_memory = s.peak;
        r.final_memory = s.mem;
        r.n_executed_ops = s.executed;
        r.n_remats = s.remats;
        r.n_evictions = s.evictions;
        r.n_eager_evictions = s.eager;
        r.n_scores = s.scores;
        r.n_nbr_visits = nbr;
        r.n_adj_visits = adj;
        r.status = s.status;
        r.failed_op = s.status == ST_OK ? -1 : s.cur_op;
        a.results[sim] = r;
    }
    __syncthreads();
}

__global__ void __launch_bounds__(WAVE) replay_kernel(KernelArgs a)
{
    const int32_t lane = threadIdx.x;
    const Slot S = slot_at(a, blockIdx.x);
    for (;;) {
        uint32_t k = 0;
        if (lane == 0) k = atomicAdd(a.queue, 1u);
        k = (uint32_t)uni((int32_t)k);
        if (k >= (uint32_t)a.n_sims) break;
        run_sim(a, a.order[k], S, lane);
    }
}

__global__ void reset_kernel(uint32_t *queue)
{
    if (threadIdx.x == 0) *queue = 0;
}

}  // namespace dtr

// launch entry used by the host library (same shared object)
extern "C" hipError_t dtr_launch_replay(const dtr::KernelArgs *args, hipStream_t stream)
{
    hipLaunchKernelGGL(dtr::reset_kernel, dim3(1), dim3(dtr::WAVE), 0, stream, args->queue);
    hipLaunchKernelGGL(dtr::replay_kernel, dim3(args->n_slots), dim3(dtr::WAVE), 0, stream, *args);
    return hipGetLastError();
}
