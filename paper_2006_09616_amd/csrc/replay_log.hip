// replay_log.hip -- gfx950 kernel of operator-log replay: DTR's eviction loop
// over storages (Appendix C.1, C.4, C.6), one wavefront per simulation.
//
// Control is wave-uniform: every lane computes the same clock, memory,
// counters and stack frame, and a state update is stored by every lane with
// the same value, so each lane later reads its own write.  Lanes work apart
// where the work is wide:
//   * the eviction search scores one storage per lane per round and reduces
//     the exact (score, id) minimum across the wave (scores N/D compared by
//     128-bit cross-multiplication, ties to the smaller storage id);
//   * h_DTR / h_{e*} / h_MSPS walk each candidate's evicted neighbourhood
//     (e* or the evicted ancestors e_R, Appendix C.2; Section 4.1) with a
//     lane-private queue and a lane-private visited bitset, cleared after
//     each walk from the queue; when the batch's largest log fits, the
//     storage states, the bitsets and the storage graph live in LDS
//     (kernel variant L), so a walk step costs LDS round trips only;
//   * h_DTR^eq keeps union-find sets of evicted storages with their running
//     cost (Appendix C.2): a node is created when a storage is evicted and
//     merged with its evicted neighbours' sets; rematerialization subtracts
//     c0 and detaches the storage (split approximation); when the node pool
//     is full it is compacted to one node per live set;
//   * an operator's inputs are checked for definedness 64 at a time, and a
//     banishing test checks a storage's dependents 64 at a time.
// Operator calls (lock inputs, define undefined inputs in listed order by
// rematerialization, allocate, run, free duplicate outputs, unlock) run on an
// explicit stack of frames in the slot; a rematerialization always calls an
// earlier operator, so the depth is bounded by the operator count.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "layout_log.h"

namespace dtr {
namespace logk {

typedef unsigned __int128 u128;

enum { ST_UNCOMPUTED = 0, ST_RESIDENT = 1, ST_EVICTED = 2, ST_BANISHED = 3 };
enum { STATUS_OK = 0, STATUS_OOM = 1, STATUS_CLOCK = 2, STATUS_CAPACITY = 3 };
enum { POLICY_EAGER = 0, POLICY_IGNORE = 1, POLICY_BANISH = 2 };
enum { SEARCH_IGNORE_SMALL = 1, SEARCH_SAMPLE = 2 };
// cost measure of a score N / (m^use_m * s^use_s)
enum { CM_ESTAR = 0, CM_EQCLASS = 1, CM_LOCAL = 2, CM_NONE = 3, CM_ANCESTORS = 4, CM_RAND = 5 };
constexpr uint64_t GOLDEN = 0x9E3779B97F4A7C15ull;
constexpr uint64_t SAMPLE_STREAM = 0xD6E8FEB86659FD93ull;

__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// workgroup control words in LDS (multi-wave workgroups): the replay index,
// the command for the helper waves, the candidate count and the e* flag of a
// walk scan
enum { CTL_K = 0, CTL_CMD = 1, CTL_N = 2, CTL_BOTH = 3 };
enum { CMD_WALK = 1, CMD_DONE = 2 };

// Order this wave's LDS and global accesses before and after (what a
// workgroup barrier gives a one-wave workgroup) without synchronizing with the
// other waves of a multi-wave workgroup.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
}
__device__ __forceinline__ int64_t uni64(int64_t v)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014)
__device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int lane_mask)
{
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, lane_mask, WAVE);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), lane_mask, WAVE);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ int64_t wave_sum(int64_t v)
{
    for (int m = WAVE / 2; m >= 1; m >>= 1) v += (int64_t)shfl64((uint64_t)v, m);
    return uni64(v);
}

// a strictly better (lower score) than b; id -1 is no candidate
__device__ __forceinline__ bool better(uint64_t na, u128 da, int32_t ia, uint64_t nb, u128 db, int32_t ib)
{
    if (ia < 0) return false;
    if (ib < 0) return true;
    const u128 l = (u128)na * db, r = (u128)nb * da;
    if (l != r) return l < r;
    return ia < ib;
}

#define GAS __attribute__((address_space(1)))
#define LAS __attribute__((address_space(3)))
// per-simulation arrays of the walks: in LDS (L) or in the slot's device memory
template <bool L, class T>
struct Ptr {
    typedef GAS T *type;
};
template <class T>
struct Ptr<true, T> {
    typedef LAS T *type;
};
template <bool L, class T>
using Mem = typename Ptr<L, T>::type;
// neighbour ids: 16 bits in LDS
template <bool L>
using Adj = typename std::conditional<L, uint16_t, int32_t>::type;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// the lowered program's tables, read with global (never flat) loads
struct ProgG {
    int32_t S, T, F, n_req;
    const GAS int64_t *s_size, *s_c0;
    const GAS uint8_t *s_const;
    const GAS int32_t *par_off, *par, *ch_off, *ch, *dt_off, *dt;
    const GAS int32_t *t_storage, *t_op;
    const GAS uint8_t *t_alias;
    const GAS int64_t *op_cost, *op_need;
    const GAS int32_t *in_off, *in, *ls_off, *ls, *out_off, *out, *rel_off, *rel, *req;
    const GAS int32_t *born_off, *born;
};

__device__ __forceinline__ ProgG prog_global(const LogProgDev &d)
{
    ProgG g;
    g.S = d.S;
    g.T = d.T;
    g.F = d.F;
    g.n_req = d.n_req;
    g.s_size = (const GAS int64_t *)d.s_size;
    g.s_c0 = (const GAS int64_t *)d.s_c0;
    g.s_const = (const GAS uint8_t *)d.s_const;
    g.par_off = (const GAS int32_t *)d.par_off;
    g.par = (const GAS int32_t *)d.par;
    g.ch_off = (const GAS int32_t *)d.ch_off;
    g.ch = (const GAS int32_t *)d.ch;
    g.dt_off = (const GAS int32_t *)d.dt_off;
    g.dt = (const GAS int32_t *)d.dt;
    g.t_storage = (const GAS int32_t *)d.t_storage;
    g.t_op = (const GAS int32_t *)d.t_op;
    g.t_alias = (const GAS uint8_t *)d.t_alias;
    g.op_cost = (const GAS int64_t *)d.op_cost;
    g.op_need = (const GAS int64_t *)d.op_need;
    g.in_off = (const GAS int32_t *)d.in_off;
    g.in = (const GAS int32_t *)d.in;
    g.ls_off = (const GAS int32_t *)d.ls_off;
    g.ls = (const GAS int32_t *)d.ls;
    g.out_off = (const GAS int32_t *)d.out_off;
    g.out = (const GAS int32_t *)d.out;
    g.rel_off = (const GAS int32_t *)d.rel_off;
    g.rel = (const GAS int32_t *)d.rel;
    g.req = (const GAS int32_t *)d.req;
    g.born_off = (const GAS int32_t *)d.born_off;
    g.born = (const GAS int32_t *)d.born;
    return g;
}

template <bool L>
struct Sim {
    ProgG P;
    Mem<L, uint8_t> state;       // storage states
    Mem<L, uint32_t> wm;         // this lane's visited bitset (walks)
    Mem<L, const int32_t> po, co;          // storage graph: parents, children
    Mem<L, const Adj<L>> pa, ca;
    // the graph that exists so far: edges per list (a prefix, lists being in
    // creation order) and each storage's cost over its tensors created so far
    Mem<L, int32_t> pcnt, ccnt;
    Mem<L, int64_t> c0d;
    // walk scan in LDS (L only): storage costs, candidate list, this lane's
    // pending stack, the candidate counter
    LAS uint16_t *cand, *stk;
    LAS uint32_t *ctr;
    LAS int64_t *rsum;         // per listed candidate: walked cost and count
    LAS int32_t *rcnt;
    LAS int32_t *ctl;          // workgroup control words (LogCtl)
    int32_t nw;                // waves in the workgroup (the others help with walks)
    int32_t wmw;               // words per visited bitset
    // slot memory
    GAS uint8_t *pinned, *pending;
    GAS int32_t *locks, *node;
    GAS int64_t *sgen, *gen;
    GAS int32_t *ufp, *ufs, *remap;
    GAS int64_t *ufc, *uft;
    GAS uint32_t *mark;        // this lane's union-find root stamps (h_DTR^eq)
    GAS int32_t *queue;        // this lane's queue
    GAS LogFrame *stack;
    Mem<L, int64_t> last;      // last access per storage
    Mem<L, const int64_t> sz;  // storage sizes
    int32_t ucap;
    // spec
    int64_t budget;
    uint64_t seed;
    int32_t policy, search, cmode;
    bool use_s, use_m, uf, walk;
    // run state (uniform)
    int64_t clock, memory, peak;
    int64_t total, base, remat_cost, executed, remats, evictions, eager;
    int64_t eviction_no, cur_op;
    int32_t status, uf_n, sp;
    // per-lane
    int32_t lane;
    uint32_t epoch;
    int64_t scores_l, nbr_l, adj_l;
};

template <bool L>
__device__ __forceinline__ bool defined(const Sim<L> &s, int32_t t)
{
    const int32_t st = s.P.t_storage[t];
    return s.state[st] == ST_RESIDENT && s.gen[t] == s.sgen[st];
}

template <bool L>
__device__ __forceinline__ bool evictable(const Sim<L> &s, int32_t st)
{
    return s.state[st] == ST_RESIDENT && s.locks[st] == 0 && !s.pinned[st] && !s.P.s_const[st];
}

// ----------------------------------------------------------- union-find --

// root of v, compressing the path (uniform: every lane stores the same links)
template <bool L>
__device__ int32_t uf_find(Sim<L> &s, int32_t v)
{
    int32_t r = v;
    for (int32_t it = 0; s.ufp[r] != r; it++) {
        if (it > s.uf_n) { s.status = STATUS_CAPACITY; return r; }
        r = s.ufp[r];
    }
    while (s.ufp[v] != r) {
        const int32_t nx = s.ufp[v];
        s.ufp[v] = r;
        v = nx;
    }
    return r;
}

// root of v without writes (lane-parallel reads)
template <bool L>
__device__ __forceinline__ int32_t uf_root(const Sim<L> &s, int32_t v)
{
    for (int32_t it = 0; it <= s.uf_n; it++) {
        const int32_t p = s.ufp[v];
        if (p == v) return v;
        v = p;
    }
    return v;
}

template <bool L>
__device__ int32_t uf_unite(Sim<L> &s, int32_t a, int32_t b)
{
    a = uf_find(s, a);
    b = uf_find(s, b);
    if (a == b) return a;
    if (s.ufs[a] < s.ufs[b]) { const int32_t t = a; a = b; b = t; }
    s.ufp[b] = a;
    s.ufs[a] += s.ufs[b];
    s.ufc[a] += s.ufc[b];
    return a;
}

// one node per live set: the sets reachable from evicted storages keep their
// cost; every evicted storage points at its set's new node
template <bool L>
__device__ void uf_compact(Sim<L> &s)
{
    const int32_t S = s.P.S, n = s.uf_n;
    for (int32_t i = s.lane; i < n; i += WAVE) s.remap[i] = 0;
    wave_sync();
    for (int32_t st = s.lane; st < S; st += WAVE)
        if (s.state[st] == ST_EVICTED) {
            const int32_t r = uf_root(s, s.node[st]);
            s.node[st] = r;
            s.remap[r] = 1;
        }
    wave_sync();
    int32_t kept = 0;
    for (int32_t b = 0; b < n; b += WAVE) {
        const int32_t i = b + s.lane;
        const bool keep = i < n && s.remap[i] != 0;
        const uint64_t m = __ballot(keep);
        if (keep) {
            const int32_t k = kept + (int32_t)__builtin_amdgcn_mbcnt_hi(
                                         (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
            s.remap[i] = k;
            s.uft[k] = s.ufc[i];
        }
        kept += __popcll(m);
    }
    wave_sync();
    for (int32_t k = s.lane; k < kept; k += WAVE) {
        s.ufc[k] = s.uft[k];
        s.ufp[k] = k;
        s.ufs[k] = 1;
    }
    for (int32_t st = s.lane; st < S; st += WAVE)
        if (s.state[st] == ST_EVICTED) s.node[st] = s.remap[s.node[st]];
    wave_sync();
    s.uf_n = uni(kept);
}

// --------------------------------------------------------------- scores --

template <bool L>
__device__ __forceinline__ uint32_t next_epoch(Sim<L> &s, int32_t used)
{
    if (++s.epoch == 0) {        // wrapped: clear this lane's stamps
        for (int32_t i = 0; i < used; i++) s.mark[i] = 0;
        s.epoch = 1;
    }
    return s.epoch;
}

// summed c0 over the evicted ancestors of x (and its evicted descendants when
// both), each storage once; the set size goes to cnt.  The visited bitset is
// clear before and after: the queue lists every storage marked.
template <bool L>
__device__ int64_t walk_cost(Sim<L> &s, int32_t x, bool both, int64_t &cnt)
{
    int64_t sum = 0;
    int32_t tail = 0;
    cnt = 0;
    for (int side = 0; side < (both ? 2 : 1); side++) {
        const auto off = side == 0 ? s.po : s.co;
        const auto adj = side == 0 ? s.pa : s.ca;
        const auto num = side == 0 ? s.pcnt : s.ccnt;
        int32_t head = tail;
        s.queue[tail++] = x;
        while (head < tail) {
            const int32_t u = s.queue[head++];
            for (int32_t e = off[u], end = off[u] + num[u]; e < end; e++) {
                const int32_t v = adj[e];
                if (s.state[v] != ST_EVICTED) continue;
                const uint32_t bit = 1u << (v & 31), w = s.wm[v >> 5];
                if (w & bit) continue;
                s.wm[v >> 5] = w | bit;
                sum += s.c0d[v];
                cnt++;
                s.queue[tail++] = v;
            }
        }
    }
    for (int32_t i = 0; i < tail; i++) {
        const int32_t v = s.queue[i];
        s.wm[v >> 5] &= ~(1u << (v & 31));
    }
    return sum;
}

// union of the sets of x's evicted parents and children, each set once
template <bool L>
__device__ int64_t eq_cost(Sim<L> &s, int32_t x, int64_t &cnt)
{
    const uint32_t ep = next_epoch(s, s.ucap);
    int64_t sum = 0;
    cnt = 0;
    for (int side = 0; side < 2; side++) {
        const auto off = side == 0 ? s.po : s.co;
        const auto adj = side == 0 ? s.pa : s.ca;
        const int32_t n = side == 0 ? s.pcnt[x] : s.ccnt[x];
        for (int32_t e = off[x]; e < off[x] + n; e++) {
            const int32_t v = adj[e];
            if (s.state[v] != ST_EVICTED) continue;
            cnt++;
            const int32_t r = uf_root(s, s.node[v]);
            if (s.mark[r] == ep) continue;
            s.mark[r] = ep;
            sum += s.ufc[r];
        }
    }
    return sum;
}

template <bool L>
__device__ __forceinline__ void score(Sim<L> &s, int32_t x, uint64_t &N, u128 &D)
{
    const int64_t m = s.sz[x];
    const int64_t stale = s.clock - s.last[x];
    const int64_t c0 = s.c0d[x];
    const int64_t deg = s.pcnt[x] + s.ccnt[x];
    int64_t cnt = 0;
    switch (s.cmode) {
    case CM_ESTAR: N = (uint64_t)(c0 + walk_cost(s, x, true, cnt)); break;
    case CM_ANCESTORS: N = (uint64_t)(c0 + walk_cost(s, x, false, cnt)); break;
    case CM_EQCLASS: N = (uint64_t)(c0 + eq_cost(s, x, cnt)); break;
    case CM_LOCAL: N = (uint64_t)c0; break;
    case CM_NONE: N = 1; break;
    default: {
        const uint64_t key = ((uint64_t)s.eviction_no << 32) + (uint64_t)(uint32_t)x;
        N = mix64(s.seed + GOLDEN * key);
        D = 1;
        return;
    }
    }
    if (s.cmode == CM_ESTAR || s.cmode == CM_ANCESTORS || s.cmode == CM_EQCLASS) {
        s.nbr_l += cnt;
        s.adj_l += deg;
    }
    D = (u128)(uint64_t)(s.use_m ? m : 1) * (u128)(uint64_t)(s.use_s ? stale : 1);
}

// ----------------------------------------------------------- eviction --

template <bool L>
__device__ void evict(Sim<L> &s, int32_t st, bool eager)
{
    if (s.uf && s.uf_n >= s.ucap) {
        uf_compact(s);
        if (s.uf_n >= s.ucap) { s.status = STATUS_CAPACITY; return; }
    }
    s.state[st] = ST_EVICTED;
    s.memory -= s.sz[st];
    if (eager) s.eager++;
    else s.evictions++;
    if (!s.uf) return;
    const int32_t nd = s.uf_n++;
    s.ufp[nd] = nd;
    s.ufs[nd] = 1;
    s.ufc[nd] = s.c0d[st];
    s.node[st] = nd;
    int32_t r = nd;
    for (int side = 0; side < 2; side++) {
        const auto off = side == 0 ? s.po : s.co;
        const auto adj = side == 0 ? s.pa : s.ca;
        const int32_t n = side == 0 ? s.pcnt[st] : s.ccnt[st];
        for (int32_t e = off[st]; e < off[st] + n; e++) {
            const int32_t v = adj[e];
            if (s.state[v] == ST_EVICTED) r = uf_unite(s, r, s.node[v]);
        }
    }
}

// The walk scan with all its data in LDS: the searched candidates are listed
// first; each lane then takes the next candidate from a shared counter as
// soon as its previous walk (and the clearing of its visited bitset) is done,
// and every iteration advances each lane's own walk by one edge, so lanes do
// not wait for the longest walk of a round.  Pending storages go on a small
// LDS stack per lane, spilling to the lane's queue in device memory; any
// order visits the same set.
// Walk the e* (or e_R) sets of the listed candidates cand[0..n): each lane
// takes the next candidate from the shared counter as soon as its previous
// walk (and the clearing of its visited bitset) has ended, and records the
// walked cost and count under the candidate's list index.
template <bool L>
__device__ void walk_candidates(Sim<L> &s, int32_t n, bool both)
{
    const int32_t W = s.wmw;
    int32_t x = -1, k = 0, e = 0, end = 0, side = 0, spl = 0, spg = 0, clr = -1;
    int64_t sum = 0;
    int32_t cnt = 0;
    auto fetch = [&]() {
        k = (int32_t)atomicAdd((uint32_t *)s.ctr, 1u);
        x = k < n ? (int32_t)s.cand[k] : -1;
        if (x >= 0) {
            side = 0;
            e = s.po[x];
            end = e + s.pcnt[x];
            sum = 0;
            cnt = 0;
        }
    };
    fetch();
    // each iteration: a finished walk clears a quad of its bitset; otherwise
    // an exhausted adjacency pops the next storage (or turns to the children,
    // or records the walk), then one edge is examined
    while (__ballot(x >= 0) != 0) {
        if (x < 0) continue;
        if (clr >= 0) {
            *(LAS u32x4 *)&s.wm[clr] = u32x4{0, 0, 0, 0};
            clr += 4;
            if (clr >= W) {
                clr = -1;
                fetch();
            }
            continue;
        }
        if (e >= end) {
            if (spl > 0 || spg > 0) {
                const int32_t u = spl > 0 ? (int32_t)s.stk[--spl] : s.queue[--spg];
                e = side == 0 ? s.po[u] : s.co[u];
                end = e + (side == 0 ? s.pcnt[u] : s.ccnt[u]);
            } else if (side == 0 && both) {
                side = 1;
                e = s.co[x];
                end = e + s.ccnt[x];
            } else {
                s.rsum[k] = sum;
                s.rcnt[k] = cnt;
                clr = 0;
                continue;
            }
        }
        if (e < end) {
            // up to two edges, their reads issued together; the two
            // neighbours are distinct (adjacency lists are sets) but may share
            // a bitset word
            const bool two = e + 1 < end;
            const auto adj = side == 0 ? s.pa : s.ca;
            const int32_t v1 = adj[e], v2 = two ? (int32_t)adj[e + 1] : v1;
            e += two ? 2 : 1;
            const uint8_t st1 = s.state[v1], st2 = s.state[v2];
            const int32_t i1 = v1 >> 5, i2 = v2 >> 5;
            const uint32_t b1 = 1u << (v1 & 31), b2 = 1u << (v2 & 31);
            const uint32_t w1 = s.wm[i1], w2 = s.wm[i2];
            const bool n1 = st1 == ST_EVICTED && !(w1 & b1);
            const bool n2 = two && st2 == ST_EVICTED && !(w2 & b2);
            if (i1 == i2) {
                if (n1 | n2) s.wm[i1] = w1 | (n1 ? b1 : 0u) | (n2 ? b2 : 0u);
            } else {
                if (n1) s.wm[i1] = w1 | b1;
                if (n2) s.wm[i2] = w2 | b2;
            }
            if (n1) {
                sum += s.c0d[v1];
                cnt++;
                if (spl < LOG_LDS_STACK) s.stk[spl++] = (uint16_t)v1;
                else s.queue[spg++] = v1;
            }
            if (n2) {
                sum += s.c0d[v2];
                cnt++;
                if (spl < LOG_LDS_STACK) s.stk[spl++] = (uint16_t)v2;
                else s.queue[spg++] = v2;
            }
        }
    }
}

template <bool L>
__device__ void scan_walk_lds(Sim<L> &s, uint64_t min_size, bool sampling, uint64_t tau, uint64_t &bn,
                              u128 &bd, int32_t &bi)
{
    const int32_t S = s.P.S;
    int32_t n = 0;
    for (int32_t b = 0; b < S; b += WAVE) {
        const int32_t x = b + s.lane;
        bool ok = false;
        if (x < S) {
            // every read issued before the first test
            const uint8_t st = s.state[x], pin = s.pinned[x], cst = s.P.s_const[x];
            const int32_t lk = s.locks[x];
            const uint64_t sz = (uint64_t)s.sz[x];
            ok = (st == ST_RESIDENT) & (lk == 0) & (pin == 0) & (cst == 0) & (sz >= min_size);
        }
        if (ok && sampling) {
            const uint64_t key = ((uint64_t)s.eviction_no << 32) + (uint64_t)(uint32_t)x;
            ok = mix64((s.seed ^ SAMPLE_STREAM) + GOLDEN * key) < tau;
        }
        const uint64_t m = __ballot(ok);
        if (ok)
            s.cand[n + (int32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                           __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0))] = (uint16_t)x;
        n += __popcll(m);
    }
    // the walks: this wave and, in a multi-wave workgroup, the helper waves
    // take candidates from the shared counter
    const bool both = s.cmode == CM_ESTAR;
    *s.ctr = 0;
    if (s.nw > 1) {
        s.ctl[CTL_CMD] = CMD_WALK;
        s.ctl[CTL_N] = n;
        s.ctl[CTL_BOTH] = both ? 1 : 0;
        __syncthreads();
    } else {
        wave_sync();
    }
    walk_candidates(s, n, both);
    if (s.nw > 1) __syncthreads();
    else wave_sync();
    // score every walked candidate
    for (int32_t q = s.lane; q < n; q += WAVE) {
        const int32_t y = s.cand[q];
        const int64_t m = s.sz[y];
        const int64_t stale = s.clock - s.last[y];
        const uint64_t N = (uint64_t)(s.c0d[y] + s.rsum[q]);
        const u128 D = (u128)(uint64_t)(s.use_m ? m : 1) * (u128)(uint64_t)(s.use_s ? stale : 1);
        if (better(N, D, y, bn, bd, bi)) { bn = N; bd = D; bi = y; }
        s.scores_l++;
        s.nbr_l += s.rcnt[q];
        s.adj_l += s.pcnt[y] + s.ccnt[y];
    }
    wave_sync();
}

// smallest r with r * r >= n
__device__ __forceinline__ uint64_t ceil_sqrt(uint64_t n)
{
    uint64_t k = (uint64_t)sqrtf((float)n);
    while (k * k < n) k++;
    while (k > 0 && (k - 1) * (k - 1) >= n) k--;
    return k;
}

// evict while memory is insufficient (Appendix C.4), under the search
// approximations when asked (Appendix E)
template <bool L>
__device__ void allocate(Sim<L> &s, int64_t need)
{
    const int32_t S = s.P.S;
    while (s.memory + need > s.budget) {
        uint64_t min_size = 0, tau = 0;
        bool sample = false;
        if (s.search) {
            int64_t n0 = 0, sum = 0;
            for (int32_t x = s.lane; x < S; x += WAVE)
                if (evictable(s, x)) { n0++; sum += s.sz[x]; }
            n0 = wave_sum(n0);
            sum = wave_sum(sum);
            if (n0 > 0 && (s.search & SEARCH_IGNORE_SMALL)) {
                const uint64_t d = 100 * (uint64_t)n0;
                min_size = ((uint64_t)sum + d - 1) / d;
            }
            if (n0 > 0 && (s.search & SEARCH_SAMPLE)) {
                const uint64_t k = ceil_sqrt((uint64_t)n0);
                if (k < (uint64_t)n0) {
                    // tau = floor(k 2^64 / n0) in two 32-bit digits
                    const uint64_t a = k << 32, q1 = a / (uint64_t)n0, r1 = a % (uint64_t)n0;
                    tau = (q1 << 32) + (r1 << 32) / (uint64_t)n0;
                    sample = true;
                }
            }
        }
        uint64_t bn = 0;
        u128 bd = 0;
        int32_t bi = -1;
        for (int pass = 0; pass < 2; pass++) {
            if (pass == 1 && !(s.search & SEARCH_SAMPLE)) break;
            const bool sampling = pass == 0 && sample;
            if constexpr (L) {
                if (s.walk) {
                    scan_walk_lds(s, min_size, sampling, tau, bn, bd, bi);
                    goto reduce;
                }
            }
            for (int32_t x = s.lane; x < S; x += WAVE) {
                if (!evictable(s, x)) continue;
                if ((uint64_t)s.sz[x] < min_size) continue;
                if (sampling) {
                    const uint64_t key = ((uint64_t)s.eviction_no << 32) + (uint64_t)(uint32_t)x;
                    if (mix64((s.seed ^ SAMPLE_STREAM) + GOLDEN * key) >= tau) continue;
                }
                uint64_t N;
                u128 D;
                score(s, x, N, D);
                s.scores_l++;
                if (better(N, D, x, bn, bd, bi)) { bn = N; bd = D; bi = x; }
            }
        reduce:
            // exact minimum across the wave
            for (int m = WAVE / 2; m >= 1; m >>= 1) {
                const uint64_t on = shfl64(bn, m);
                const uint64_t dlo = shfl64((uint64_t)bd, m), dhi = shfl64((uint64_t)(bd >> 64), m);
                const int32_t oi = __shfl_xor(bi, m, WAVE);
                const u128 od = ((u128)dhi << 64) | dlo;
                if (better(on, od, oi, bn, bd, bi)) { bn = on; bd = od; bi = oi; }
            }
            bi = uni(bi);
            if (bi >= 0) break;
        }
        if (bi < 0) { s.status = STATUS_OOM; return; }
        evict(s, bi, false);
        if (s.status) return;
        s.eviction_no++;
    }
}

// ----------------------------------------------------------- policies --

// Banish st if no operator holds it and every tensor computed from it
// (outside it) is defined or gone; pin those tensors' resident storages.
// Otherwise st stays pending (Appendix C.4, C.5).
template <bool L>
__device__ void try_banish(Sim<L> &s, int32_t st)
{
    const int32_t b = s.P.dt_off[st], e = s.P.dt_off[st + 1];
    bool blocked = s.locks[st] > 0;
    for (int32_t q = b; q < e && !blocked; q += WAVE) {
        bool bad = false;
        if (q + s.lane < e) {
            const int32_t v = s.P.dt[q + s.lane];
            bad = !defined(s, v) && s.state[s.P.t_storage[v]] != ST_BANISHED;
        }
        blocked = __ballot(bad) != 0;
    }
    if (blocked) { s.pending[st] = 1; return; }
    s.pending[st] = 0;
    if (s.state[st] == ST_RESIDENT) s.memory -= s.sz[st];
    s.state[st] = ST_BANISHED;
    s.eager++;
    for (int32_t q = b + s.lane; q < e; q += WAVE) {
        const int32_t d = s.P.t_storage[s.P.dt[q]];
        if (s.state[d] == ST_RESIDENT) s.pinned[d] = 1;
    }
    wave_sync();
}

template <bool L>
__device__ void release(Sim<L> &s, int32_t st)
{
    if (s.policy == POLICY_EAGER) {
        if (evictable(s, st)) evict(s, st, true);
    } else if (s.policy == POLICY_BANISH) {
        try_banish(s, st);
    }
}

// ---------------------------------------------------------- operators --

template <bool L>
__device__ void push(Sim<L> &s, int32_t o, int32_t remat)
{
    if (s.sp >= s.P.F + 2) { s.status = STATUS_CAPACITY; return; }
    for (int32_t e = s.P.ls_off[o]; e < s.P.ls_off[o + 1]; e++) s.locks[s.P.ls[e]] += 1;
    GAS LogFrame *f = &s.stack[s.sp];
    f->op = o;
    f->next = s.P.in_off[o];
    f->remat = remat;
    f->pad = 0;
    s.sp++;
}

// run operator o once its inputs are defined: allocate its new storages, run,
// free the copies of outputs already defined, unlock (Appendix C.4)
template <bool L>
__device__ void execute(Sim<L> &s, int32_t o, bool remat)
{
    const int64_t need = s.P.op_need[o];
    allocate(s, need);
    if (s.status) return;
    const int32_t ib = s.P.in_off[o], ie = s.P.in_off[o + 1];
    const int32_t ob = s.P.out_off[o], oe = s.P.out_off[o + 1];
    for (int32_t e = s.P.ls_off[o]; e < s.P.ls_off[o + 1]; e++) s.last[s.P.ls[e]] = s.clock;
    for (int32_t q = ob; q < oe; q++) s.last[s.P.t_storage[s.P.out[q]]] = s.clock;
    const int64_t c = s.P.op_cost[o];
    s.clock += c;
    s.total += c;
    s.executed++;
    if (remat) { s.remats++; s.remat_cost += c; }
    else s.base += c;
    s.memory += need;
    if (s.memory > s.peak) s.peak = s.memory;
    for (int32_t q = ob; q < oe; q++) {
        const int32_t v = s.P.out[q];
        if (s.P.t_alias[v]) continue;
        const int32_t st = s.P.t_storage[v];
        const uint8_t was = s.state[st];
        if (was == ST_RESIDENT) { s.memory -= s.sz[st]; continue; }
        s.state[st] = ST_RESIDENT;
        const int64_t g = s.sgen[st] + 1;
        s.sgen[st] = g;
        s.gen[v] = g;
        if (s.uf && was == ST_EVICTED) {
            const int32_t r = uf_find(s, s.node[st]);
            s.ufc[r] -= s.c0d[st];
            s.node[st] = -1;
        }
    }
    for (int32_t q = ob; q < oe; q++) {
        const int32_t v = s.P.out[q];
        if (s.P.t_alias[v]) s.gen[v] = s.sgen[s.P.t_storage[v]];
    }
    if (!remat) {
        // the operator's first run creates its tensors: their costs join
        // their storages' and their edges join the graph (Appendix C.2)
        for (int32_t q = ob; q < oe; q++) {
            const int32_t st = s.P.t_storage[s.P.out[q]];
            if (!s.P.s_const[st]) s.c0d[st] += c;
        }
        for (int32_t b = s.P.born_off[o]; b < s.P.born_off[o + 1]; b++) {
            const int32_t par = s.P.born[2 * b], st = s.P.born[2 * b + 1];
            s.pcnt[st] += 1;
            s.ccnt[par] += 1;
        }
    }
    if (s.clock >= CLOCK_LIMIT) { s.status = STATUS_CLOCK; return; }
    for (int32_t e = s.P.ls_off[o]; e < s.P.ls_off[o + 1]; e++) s.locks[s.P.ls[e]] -= 1;
    if (remat && s.policy == POLICY_BANISH)
        for (int32_t e = ib; e < ie; e++) {
            const int32_t st = s.P.t_storage[s.P.in[e]];
            if (s.pending[st]) try_banish(s, st);
        }
}

// call operator o (a rematerialization if remat), defining undefined inputs
// first, in listed order, by calling their operators
template <bool L>
__device__ void call(Sim<L> &s, int32_t o, int32_t remat)
{
    const int32_t floor = s.sp;
    push(s, o, remat);
    while (s.sp > floor && !s.status) {
        const GAS LogFrame *top = &s.stack[s.sp - 1];
        const int32_t f_op = top->op, f_next = top->next, f_remat = top->remat;
        const int32_t end = s.P.in_off[f_op + 1];
        int32_t found = -1;
        for (int32_t e = f_next; e < end; e += WAVE) {
            const int32_t i = e + s.lane;
            const bool undef = i < end && !defined(s, s.P.in[i]);
            const uint64_t m = __ballot(undef);
            if (m) { found = e + (int32_t)__builtin_ctzll(m); break; }
        }
        found = uni(found);
        if (found >= 0) {
            s.stack[s.sp - 1].next = found + 1;
            push(s, s.P.t_op[s.P.in[found]], 1);
            continue;
        }
        execute(s, f_op, f_remat != 0);
        if (s.status) return;
        s.sp--;
    }
}

template <bool L>
__device__ void run_sim(const LogKernelArgs &a, int32_t sim, uint8_t *base, int32_t lane, uint8_t *lds, int32_t nw)
{
    Sim<L> s;
    const SpecDev sp = a.specs[sim];
    s.P = prog_global(a.progs[sp.trace]);
    const LogSlotLayout &Y = a.L;
    GAS uint8_t *gb = (GAS uint8_t *)base;
    s.pinned = gb + Y.pinned;
    s.pending = gb + Y.pending;
    s.locks = (GAS int32_t *)(gb + Y.locks);
    s.node = (GAS int32_t *)(gb + Y.node);
    s.sgen = (GAS int64_t *)(gb + Y.sgen);
    s.gen = (GAS int64_t *)(gb + Y.gen);
    s.ufp = (GAS int32_t *)(gb + Y.uf_parent);
    s.ufs = (GAS int32_t *)(gb + Y.uf_size);
    s.remap = (GAS int32_t *)(gb + Y.uf_remap);
    s.ufc = (GAS int64_t *)(gb + Y.uf_cost);
    s.uft = (GAS int64_t *)(gb + Y.uf_tmp);
    s.mark = (GAS uint32_t *)(gb + Y.mark) + (size_t)lane * (size_t)Y.mcap;
    s.queue = (GAS int32_t *)(gb + Y.queue) + (size_t)lane * (size_t)(Y.S_max + 2);
    s.stack = (GAS LogFrame *)(gb + Y.stack);
    s.ucap = (int32_t)Y.ucap;
    const int32_t W = a.wm_words;
    s.wmw = W;
    s.nw = nw;
    s.ctl = nullptr;
    if constexpr (L) {
        s.state = (Mem<L, uint8_t>)(lds + a.lds_state);
        s.wm = (Mem<L, uint32_t>)(lds + a.lds_wm) + lane * W;
        s.po = (Mem<L, const int32_t>)(lds + a.lds_po);
        s.co = (Mem<L, const int32_t>)(lds + a.lds_co);
        s.pa = (Mem<L, const Adj<L>>)(lds + a.lds_pa);
        s.ca = (Mem<L, const Adj<L>>)(lds + a.lds_ca);
        s.c0d = (Mem<L, int64_t>)(lds + a.lds_c0);
        s.pcnt = (Mem<L, int32_t>)(lds + a.lds_pcnt);
        s.ccnt = (Mem<L, int32_t>)(lds + a.lds_ccnt);
        s.cand = (LAS uint16_t *)(lds + a.lds_cand);
        s.stk = (LAS uint16_t *)(lds + a.lds_stk) + lane * LOG_LDS_STACK;
        s.ctr = (LAS uint32_t *)(lds + a.lds_ctr);
        s.rsum = (LAS int64_t *)(lds + a.lds_rsum);
        s.rcnt = (LAS int32_t *)(lds + a.lds_rcnt);
        s.ctl = (LAS int32_t *)(lds + a.lds_ctl);
        s.last = (Mem<L, int64_t>)(lds + a.lds_last);
        s.sz = (Mem<L, const int64_t>)(lds + a.lds_sz);
    } else {
        s.state = (Mem<L, uint8_t>)(base + Y.state);
        s.wm = (Mem<L, uint32_t>)(base + Y.wmark) + lane * W;
        s.po = (Mem<L, const int32_t>)s.P.par_off;
        s.co = (Mem<L, const int32_t>)s.P.ch_off;
        s.pa = (Mem<L, const Adj<L>>)s.P.par;
        s.ca = (Mem<L, const Adj<L>>)s.P.ch;
        s.last = (Mem<L, int64_t>)(gb + Y.last);
        s.sz = s.P.s_size;
        s.c0d = (Mem<L, int64_t>)(gb + Y.c0d);
        s.pcnt = (Mem<L, int32_t>)(gb + Y.pcnt);
        s.ccnt = (Mem<L, int32_t>)(gb + Y.ccnt);
    }
    s.budget = sp.budget;
    s.seed = sp.seed;
    s.policy = sp.policy;
    s.search = sp.search;
    const int32_t h = sp.heuristic;
    if (h >= 16) {
        const int32_t f = h - 16;
        s.cmode = f >> 2;
        s.use_s = (f & 2) != 0;
        s.use_m = (f & 1) != 0;
    } else {
        // h_DTR, h_DTR^eq, h_DTR^local, h_LRU, h_size, h_rand, h_{e*}, h_MSPS:
        // cost measure (a nibble each), staleness used, size used
        constexpr uint32_t CM = (CM_ESTAR << 0) | (CM_EQCLASS << 4) | (CM_LOCAL << 8) | (CM_NONE << 12) |
                                (CM_NONE << 16) | (CM_RAND << 20) | (CM_ESTAR << 24) | ((uint32_t)CM_ANCESTORS << 28);
        constexpr uint32_t US = 0x0F, UM = 0xD7;
        const int32_t i = h & 7;
        s.cmode = (int32_t)((CM >> (4 * i)) & 0xF);
        s.use_s = ((US >> i) & 1) != 0;
        s.use_m = ((UM >> i) & 1) != 0;
    }
    s.uf = s.cmode == CM_EQCLASS;
    s.walk = s.cmode == CM_ESTAR || s.cmode == CM_ANCESTORS;
    s.lane = lane;
    s.epoch = 0;
    s.scores_l = s.nbr_l = s.adj_l = 0;
    s.clock = s.memory = s.peak = 0;
    s.total = s.base = s.remat_cost = s.executed = s.remats = s.evictions = s.eager = 0;
    s.eviction_no = s.cur_op = 0;
    s.status = STATUS_OK;
    s.uf_n = 0;
    s.sp = 0;

    const int32_t S = s.P.S, T = s.P.T, F = s.P.F;
    for (int32_t i = lane; i < S; i += WAVE) {
        s.state[i] = ST_UNCOMPUTED;
        s.pinned[i] = s.P.s_const[i];
        s.pending[i] = 0;
        s.locks[i] = 0;
        s.node[i] = -1;
        s.sgen[i] = 0;
        s.last[i] = 0;
        s.c0d[i] = 0;
        s.pcnt[i] = 0;
        s.ccnt[i] = 0;
    }
    for (int32_t i = lane; i < T; i += WAVE) s.gen[i] = -1;
    if (s.uf) {
        GAS uint32_t *M = (GAS uint32_t *)(gb + Y.mark);
        for (int32_t l = 0; l < WAVE; l++)
            for (int32_t i = lane; i < s.ucap; i += WAVE) M[(size_t)l * (size_t)Y.mcap + i] = 0;
    }
    if (s.walk) {
        Mem<L, uint32_t> M = s.wm - lane * W;
        for (int32_t i = lane; i < WAVE * W; i += WAVE) M[i] = 0;
    }
    if constexpr (L) {
        // the storage graph of this log, 16-bit neighbour ids
        Mem<L, int32_t> po = (Mem<L, int32_t>)s.po, co = (Mem<L, int32_t>)s.co;
        Mem<L, Adj<L>> pa = (Mem<L, Adj<L>>)s.pa, ca = (Mem<L, Adj<L>>)s.ca;
        for (int32_t i = lane; i <= S; i += WAVE) {
            po[i] = s.P.par_off[i];
            co[i] = s.P.ch_off[i];
        }
        const int32_t E = s.P.par_off[S];
        for (int32_t e = lane; e < E; e += WAVE) {
            pa[e] = (Adj<L>)s.P.par[e];
            ca[e] = (Adj<L>)s.P.ch[e];
        }
        Mem<L, int64_t> szl = (Mem<L, int64_t>)s.sz;
        for (int32_t i = lane; i < S; i += WAVE) szl[i] = s.P.s_size[i];
    }
    wave_sync();

    for (int32_t o = 0; o < F && !s.status; o++) {
        s.cur_op = o;
        call(s, o, 0);
        if (s.status) break;
        for (int32_t e = s.P.rel_off[o]; e < s.P.rel_off[o + 1] && !s.status; e++) release(s, s.P.rel[e]);
    }
    if (!s.status) {
        // output condition: every tensor still referenced is defined and held
        s.cur_op = F;
        for (int32_t k = 0; k < s.P.n_req && !s.status; k++) {
            const int32_t t = s.P.req[k];
            s.locks[s.P.t_storage[t]] += 1;
            if (!defined(s, t)) call(s, s.P.t_op[t], 1);
        }
    }
    const int64_t scores = wave_sum(s.scores_l), nbr = wave_sum(s.nbr_l), adj = wave_sum(s.adj_l);
    if (lane == 0) {
        ResultDev r;
        r.total_cost = s.total;
        r.base_cost = s.base;
        r.remat_cost = s.remat_cost;
        r.peak_memory = s.peak;
        r.final_memory = s.memory;
        r.n_executed_ops = s.executed;
        r.n_remats = s.remats;
        r.n_evictions = s.evictions;
        r.n_eager_evictions = s.eager;
        r.n_scores = scores;
        r.n_nbr_visits = nbr;
        r.n_adj_visits = adj;
        r.status = s.status;
        r.failed_op = s.status == STATUS_OK ? -1 : (int32_t)s.cur_op;
        a.results[sim] = r;
    }
    if (nw > 1) {
        // release the helper waves from this replay
        s.ctl[CTL_CMD] = CMD_DONE;
        __syncthreads();
    } else {
        wave_sync();
    }
}

// A helper wave of a multi-wave workgroup: joins the replaying wave's walk
// scans (one workgroup barrier before, one after each) until it is released.
// Each of its lanes has its own visited bitset, LDS stack and global queue.
template <bool L>
__device__ void help_walks(const LogKernelArgs &a, uint8_t *base, int32_t lane, int32_t wave, uint8_t *lds)
{
    if constexpr (L) {
        Sim<L> s;
        const LogSlotLayout &Y = a.L;
        GAS uint8_t *gb = (GAS uint8_t *)base;
        const int32_t W = a.wm_words, id = wave * WAVE + lane;
        s.wmw = W;
        s.lane = lane;
        s.state = (Mem<L, uint8_t>)(lds + a.lds_state);
        s.wm = (Mem<L, uint32_t>)(lds + a.lds_wm) + id * W;
        s.po = (Mem<L, const int32_t>)(lds + a.lds_po);
        s.co = (Mem<L, const int32_t>)(lds + a.lds_co);
        s.pa = (Mem<L, const Adj<L>>)(lds + a.lds_pa);
        s.ca = (Mem<L, const Adj<L>>)(lds + a.lds_ca);
        s.c0d = (Mem<L, int64_t>)(lds + a.lds_c0);
        s.pcnt = (Mem<L, int32_t>)(lds + a.lds_pcnt);
        s.ccnt = (Mem<L, int32_t>)(lds + a.lds_ccnt);
        s.cand = (LAS uint16_t *)(lds + a.lds_cand);
        s.stk = (LAS uint16_t *)(lds + a.lds_stk) + id * LOG_LDS_STACK;
        s.ctr = (LAS uint32_t *)(lds + a.lds_ctr);
        s.rsum = (LAS int64_t *)(lds + a.lds_rsum);
        s.rcnt = (LAS int32_t *)(lds + a.lds_rcnt);
        s.queue = (GAS int32_t *)(gb + Y.queue) + (size_t)id * (size_t)(Y.S_max + 2);
        const LAS int32_t *ctl = (const LAS int32_t *)(lds + a.lds_ctl);
        for (;;) {
            __syncthreads();
            if (ctl[CTL_CMD] == CMD_DONE) break;
            walk_candidates(s, ctl[CTL_N], ctl[CTL_BOTH] != 0);
            __syncthreads();
        }
    }
}

// One replay per workgroup at a time.  In the LDS variant the workgroup may
// hold helper waves (a.waves in all) that join the replaying wave's walk scans;
// every wave learns the next replay from the control words after a workgroup
// barrier, so all of them leave the loop together.
template <bool L>
__global__ void __launch_bounds__(L ? MAX_LOG_WAVES * WAVE : WAVE) log_kernel(LogKernelArgs a)
{
    extern __shared__ uint8_t lds_dyn[];
    const int32_t lane = (int32_t)threadIdx.x & (WAVE - 1);
    const int32_t wave = uni((int32_t)threadIdx.x / WAVE);
    const int32_t nw = L ? a.waves : 1;
    uint8_t *base = a.slots + (size_t)blockIdx.x * (size_t)a.L.bytes;
    LAS int32_t *ctl = (LAS int32_t *)(lds_dyn + a.lds_ctl);
    if constexpr (L) {
        if (wave > 0) {
            // a helper's visited bitsets start clear (each walk clears its own)
            LAS uint32_t *M = (LAS uint32_t *)(lds_dyn + a.lds_wm) + (size_t)wave * WAVE * a.wm_words;
            for (int32_t i = lane; i < WAVE * a.wm_words; i += WAVE) M[i] = 0;
        }
    }
    for (;;) {
        uint32_t k = 0;
        if (wave == 0 && lane == 0) k = atomicAdd(a.queue, 1u);
        if (nw > 1) {
            if (wave == 0 && lane == 0) ctl[CTL_K] = (int32_t)k;
            __syncthreads();
            k = (uint32_t)uni(ctl[CTL_K]);
        } else {
            k = (uint32_t)uni((int32_t)k);
        }
        if (k >= (uint32_t)a.n_sims) break;
        if (wave == 0) run_sim<L>(a, a.order[k], base, lane, lds_dyn, nw);
        else help_walks<L>(a, base, lane, wave, lds_dyn);
    }
}

__global__ void log_reset_kernel(uint32_t *queue)
{
    if (threadIdx.x == 0) queue[0] = 0;
}

}  // namespace logk
}  // namespace dtr

// Launch entry used by the host library (same shared object).
extern "C" hipError_t dtr_launch_log(const dtr::LogKernelArgs *args, hipStream_t stream)
{
    using namespace dtr;
    hipLaunchKernelGGL(logk::log_reset_kernel, dim3(1), dim3(WAVE), 0, stream, args->queue);
    if (args->n_sims > 0) {
        if (args->lds_bytes > 0) {
            if (args->lds_bytes > 64 * 1024) {
                hipError_t e = hipFuncSetAttribute((const void *)logk::log_kernel<true>,
                                                   hipFuncAttributeMaxDynamicSharedMemorySize, args->lds_bytes);
                if (e != hipSuccess) return e;
            }
            hipLaunchKernelGGL(logk::log_kernel<true>, dim3(args->n_slots), dim3(WAVE * args->waves), args->lds_bytes,
                               stream, *args);
        }
        else
            hipLaunchKernelGGL(logk::log_kernel<false>, dim3(args->n_slots), dim3(WAVE), 0, stream, *args);
    }
    return hipGetLastError();
}
