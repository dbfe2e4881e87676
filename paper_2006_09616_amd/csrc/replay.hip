// replay.hip -- gfx950 kernels of the batched DTR eviction-loop simulator.
//
// One wavefront (64 lanes, one workgroup) owns one simulation at a time and
// pulls the next one from a global work counter (persistent grid, longest
// traces first).  DTR's operator call (Section 2; Appendix C.4) is a chain of
// dependent steps, so the kernel is organised around memory latency: every
// step is arranged so that independent reads are issued together and the
// number of dependent memory round trips per operation stays small.
//
//  * wave-uniform control: clock, memory, counters and the current frame are
//    identical in every lane; read-only trace tables are read through the
//    scalar cache (one 32-byte record per tensor);
//  * lane-parallel bookkeeping: the inputs of an operation are locked,
//    checked and unlocked by one lane each, with their state kept in
//    registers for the life of the frame; release lists are checked in
//    parallel;
//  * the evictable pool (Appendix C.4 "Runtime state") is a tombstoned
//    array of 64-byte slots read as coalesced quads; each lane scores one or two candidates per
//    round with all slot reads issued at once, and the exact (score, id)
//    minimum is reduced across lanes;
//  * h_DTR^eq (Appendix C.2): each pool slot caches the union-find nodes of
//    its candidate's evicted neighbours, kept current as neighbours are
//    evicted and rematerialized, so a score needs one dependent node read
//    (two if the node is no longer a root); union-find nodes are created at
//    eviction and carry the running cost of their set; all sets adjacent to
//    an evicted tensor are found in parallel and merged at once;
//    rematerialization subtracts c0 and detaches the tensor (split
//    approximation); the node pool is compacted when full;
//  * h_DTR / h_{e*}: each lane walks its candidate's evicted ancestors and
//    descendants (e*, Appendix C.2) with lane-private epoch stamps, taking the
//    next candidate as soon as its walk ends.
//
// Scores N/D are compared exactly by 128-bit cross-multiplication; ties go to
// the smaller tensor id.  Last-access times are not kept per tensor: a tensor
// joins the pool right after the operation that last referenced it, so the
// pool slot receives that operation's start time.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/dtr_sim.h"
#include "layout.h"

namespace dtr {

typedef unsigned __int128 u128;

enum { H_DTR = 0, H_EQ = 1, H_LOCAL = 2, H_LRU = 3, H_SIZE = 4, H_RAND = 5, H_ESTAR = 6, H_MSPS = 7,
       H_FAMILY = 16 };
// cost measure of a score N / (m^use_m * s^use_s): c0 + e* cost, c0 +
// union-find neighbourhood cost, c0, 1, c0 + e_R cost (evicted ancestors
// only), or a random draw
enum { CM_ESTAR = 0, CM_EQCLASS = 1, CM_LOCAL = 2, CM_NONE = 3, CM_ANCESTORS = 4, CM_RAND = 5 };
enum { ST_OK = 0, ST_OOM = 1, ST_CLOCK = 2, ST_CAPACITY = 3 };

// state word values (low 32 bits of a tensor's state); >= 0: evicted (node)
constexpr int32_t S_BANISHED = -5;    // freed for good (banishing policy)
constexpr int32_t S_PINNED = -4;      // resident, never evictable: a banished tensor's child
constexpr int32_t S_CONST = -3;
constexpr int32_t S_UNCOMPUTED = -2;
constexpr int32_t S_RESIDENT = -1;
enum { POLICY_EAGER = 0, POLICY_IGNORE = 1, POLICY_BANISH = 2 };
enum { SEARCH_IGNORE_SMALL = 1, SEARCH_SAMPLE = 2 };
// lock counts of 255 and more live in the slot's lockx array (the 8-bit field
// then reads LOCKS_SAT)
constexpr uint32_t LOCKS_SAT = 255;
constexpr uint8_t FLAG_CONST = 1;
constexpr int K = NB_CACHE;
constexpr int KQ = K / 4;        // 16-byte quads of cached nodes per pool slot
constexpr int PQ = (int)(sizeof(PoolSlot) / 16);   // quads per pool slot
static_assert(K % 4 == 0 && PQ == 2 + KQ, "pool slot: two header quads, then the cache");
constexpr int LB = 8;            // neighbour reads issued together when building a cache
static_assert(LB == NB_HEAD, "a cache build may take its first chunk from the record element");
// kernel specialisations by heuristic class (register budgets differ widely),
// each with exact search or with the search approximations (HC | HC_APPROX)
enum { HC_EQ = 0, HC_WALK = 1, HC_SIMPLE = 2, HC_APPROX = 4 };
__host__ __device__ constexpr int cls(int hc) { return hc & 3; }
__host__ __device__ constexpr bool approx(int hc) { return (hc & HC_APPROX) != 0; }
// candidates per lane per scan round (their reads are issued together); the
// h_DTR^eq round is instruction-issue bound, so a second candidate per lane
// only doubles the round
template <int HC>
struct Round {
    static constexpr int value = cls(HC) == HC_EQ ? 1 : 2;
    static_assert(POOL_LDS % (WAVE * value) == 0, "a scan round lies wholly in LDS or wholly in global memory");
};

// ------------------------------------------------------------- helpers --

__device__ __forceinline__ int32_t uni(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ int64_t uni64(int64_t v)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// lane j's value (j wave-uniform)
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int32_t j)
{
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, j);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), j);
    return ((uint64_t)hi << 32) | lo;
}

#define GAS __attribute__((address_space(1)))    // global memory
#define LAS __attribute__((address_space(3)))    // LDS
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// read-only trace tables: constant address space, so uniform reads become
// scalar loads
template <class T>
__device__ __forceinline__ T cld(const T *p) { return *(const __attribute__((address_space(4))) T *)p; }
// per-lane reads of the same tables: global loads (never flat)
template <class T>
__device__ __forceinline__ T gld(const T *p) { return *(const GAS T *)p; }

__device__ __forceinline__ int32_t lane_rank(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

__device__ __forceinline__ uint64_t ts_make(int32_t sw, uint32_t pos, uint32_t locks)
{
    return (uint64_t)(uint32_t)sw | ((uint64_t)(pos & 0xFFFFFFu) << 32) | ((uint64_t)locks << 56);
}
__device__ __forceinline__ int32_t ts_sw(uint64_t w) { return (int32_t)(uint32_t)w; }
__device__ __forceinline__ uint32_t ts_pos(uint64_t w) { return (uint32_t)(w >> 32) & 0xFFFFFFu; }
__device__ __forceinline__ uint32_t ts_locks(uint64_t w) { return (uint32_t)(w >> 56); }
__device__ __forceinline__ bool ts_in_pool(uint64_t w) { return ts_sw(w) == S_RESIDENT && ts_locks(w) == 0; }

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

// Union-find node store: ids below UF_LDS in this wavefront's LDS array, the
// rest in the slot's global array; one id space, read through flat pointers
// (or straight from LDS while every node id is below UF_LDS).
struct NodeStore {
    UfNode *lds;
    LAS UfNode *lds_l;
    UfNode *glob;
    __device__ __forceinline__ UfNode &operator[](int32_t id) const
    {
        return id < UF_LDS ? lds[id] : glob[id - UF_LDS];
    }
};

// LDS pool slots are padded to 80 bytes, so the 16-byte reads of 64
// consecutive slots fall in distinct bank groups
constexpr int PQL = PQ + 1;
struct __attribute__((aligned(16))) PoolSlotL {
    PoolSlot s;
    i32x4 pad;
};
// Evictable pool: slots below POOL_LDS in this wavefront's LDS array, the
// rest in the slot's global array (same indices).
struct Slot {
    GAS uint64_t *tst;
    GAS int32_t *lockx;           // lock counts >= LOCKS_SAT
    PoolSlotL *lpool;             // flat view of the LDS head
    LAS PoolSlotL *lpool_l;
    GAS PoolSlot *gpool;
    NodeStore nodes;
    GAS int32_t *remap;
    GAS i32x4 *stack;             // StackFrame records, three quads each
    GAS uint8_t *visb;            // walk heuristics: lane-private visited flags (a byte per tensor)
    GAS int32_t *wq;              // and member queues
    GAS uint32_t *bigvis;         // each wavefront's bitmap and queue for large walks
    GAS int32_t *bigq;
    GAS int32_t *ovf;             // pool slots of the candidates whose walk is large
    GAS uint8_t *pending;         // released, banishing deferred (banishing policy)
    int32_t pcap, ucap, n_max;
    int32_t vis_words, vis_bytes, wq_cap;
    __device__ __forceinline__ PoolSlot &pool(int32_t i) const
    {
        return i < POOL_LDS ? lpool[i].s : *(PoolSlot *)(gpool + i);
    }
};

__device__ __forceinline__ Slot slot_at(const KernelArgs &a, int32_t k)
{
    uint8_t *b = a.slots + (size_t)k * (size_t)a.L.bytes;
    Slot S;
    S.tst = (GAS uint64_t *)(b + a.L.tst);
    S.lockx = (GAS int32_t *)(b + a.L.lockx);
    S.lpool = nullptr;
    S.lpool_l = nullptr;
    S.gpool = (GAS PoolSlot *)(b + a.L.pool);
    S.nodes.lds = nullptr;
    S.nodes.lds_l = nullptr;
    S.nodes.glob = (UfNode *)(b + a.L.nodes);
    S.remap = (GAS int32_t *)(b + a.L.uf_remap);
    S.stack = (GAS i32x4 *)(b + a.L.stack);
    S.visb = (GAS uint8_t *)(b + a.L.vis);
    S.wq = (GAS int32_t *)(b + a.L.wq);
    S.bigvis = (GAS uint32_t *)(b + a.L.bigvis);
    S.bigq = (GAS int32_t *)(b + a.L.bigq);
    S.ovf = (GAS int32_t *)(b + a.L.ovf);
    S.pending = (GAS uint8_t *)(b + a.L.pending);
    S.pcap = (int32_t)a.L.pcap;
    S.ucap = (int32_t)a.L.ucap;
    S.n_max = (int32_t)a.L.n_max;
    S.vis_words = (int32_t)a.L.vis_words;
    S.vis_bytes = (int32_t)a.L.vis_bytes;
    S.wq_cap = (int32_t)a.L.wq_cap;
    return S;
}

// Wave-uniform simulation state.
struct Sim {
    TraceDev t;
    Slot S;
    int32_t h;
    int32_t cmode, use_s, use_m;  // the heuristic as (cost measure, staleness used, size used)
    int32_t policy;               // what a release does
    int32_t search;               // search approximation flags
    int32_t lane;
    int64_t budget;
    uint64_t seed;
    int64_t T, mem, peak;
    int32_t pool_end, pool_live;
    int32_t uf_n, uf_limit;      // nodes in use; count that triggers a compaction
    int32_t status, cur_op;
    int32_t nw;                   // wavefronts in the workgroup (walk heuristics)
    int32_t trace_idx;
    LAS struct WalkCtl *ctl;      // their control block in LDS
    unsigned long long *progress; // the launch's progress counter (walk heuristics)
    int64_t evict_no;
    int64_t total, base, remat_cost, executed, remats, evictions, eager, scores;
    int64_t nbr, adj;     // per-lane partial sums, reduced at the end
#ifdef DTR_PROFILE
    int64_t prof_scan_cycles, prof_scans, prof_rounds;
    int64_t prof_slow, prof_global_nodes, prof_uf_compact, prof_pool_compact;
    int64_t prof_ph[PROF_PHASES];
#endif
};

// phase timers (DTR_PROFILE builds only)
#ifdef DTR_PROFILE
#define PROF_T0(v) const int64_t v = (int64_t)__builtin_readcyclecounter()
#define PROF_ADD(k, v) s.prof_ph[k] += (int64_t)__builtin_readcyclecounter() - (v)
#else
#define PROF_T0(v)
#define PROF_ADD(k, v)
#endif
enum { PH_EVICT = 0, PH_EXECUTE, PH_UNLOCK, PH_LOCK, PH_RELEASE, PH_RESUME, PH_OUTPUT, PH_DESCEND };

__device__ __forceinline__ void set_status(Sim &s, int32_t st)
{
    if (s.status == ST_OK) s.status = st;
}

// uniform read of a tensor's static record (two 16-byte scalar loads)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ TRec rec_u(const Sim &s, int32_t x)
{
    const __attribute__((address_space(4))) u32x4 *p =
        (const __attribute__((address_space(4))) u32x4 *)&s.t.rec[x].r;
    const u32x4 a = p[0], b = p[1];
    TRec r;
    r.size = (int64_t)((uint64_t)a.x | ((uint64_t)a.y << 32));
    r.c0 = (int32_t)a.z;
    r.producer = (int32_t)a.w;
    r.in_b = (int32_t)b.x;
    r.in_e = (int32_t)b.y;
    r.adj_b = (int32_t)b.z;
    r.adj_e = (int32_t)b.w;
    return r;
}

// per-lane read of a tensor's static record (two 16-byte global loads)
__device__ __forceinline__ TRec rec_v_t(const TraceDev &t, int32_t x)
{
    const GAS u32x4 *p = (const GAS u32x4 *)&t.rec[x].r;
    const u32x4 a = p[0], b = p[1];
    TRec r;
    r.size = (int64_t)((uint64_t)a.x | ((uint64_t)a.y << 32));
    r.c0 = (int32_t)a.z;
    r.producer = (int32_t)a.w;
    r.in_b = (int32_t)b.x;
    r.in_e = (int32_t)b.y;
    r.adj_b = (int32_t)b.z;
    r.adj_e = (int32_t)b.w;
    return r;
}

__device__ __forceinline__ TRec rec_v(const Sim &s, int32_t x) { return rec_v_t(s.t, x); }

// ------------------------------------------------------ neighbour cache --

// This lane's cache of evicted-neighbour nodes for a tensor with neighbour
// range [b, e), built in registers: the first K evicted neighbours' nodes
// (unused entries hold node 0, the null node: cost 0, its own root).  Returns
// the cache; `deg` receives (degree << 8) | count (K + 1: overflowed).
// Neighbour states are read LB at a time, all loads unconditional.
struct NbCache {
    i32x4 q[KQ];
};

__device__ __forceinline__ NbCache list_build(const Sim &s, int32_t b, int32_t e, int32_t &deg,
                                              const i32x4 *head = nullptr)
{
    int32_t c[K];
#pragma unroll
    for (int k = 0; k < K; k++) c[k] = 0;
    int32_t cnt = 0;
    for (int32_t k0 = b; k0 < e; k0 += LB) {
        int32_t w[LB];
        int32_t q[LB];
        if (head && k0 == b) {
#pragma unroll
            for (int j = 0; j < LB / 4; j++) {
                w[4 * j] = head[j].x;
                w[4 * j + 1] = head[j].y;
                w[4 * j + 2] = head[j].z;
                w[4 * j + 3] = head[j].w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < LB; j++) w[j] = gld(s.t.adj + (k0 + j < e ? k0 + j : k0));
        }
#pragma unroll
        for (int j = 0; j < LB; j++) q[j] = ts_sw(s.S.tst[w[j]]);
#pragma unroll
        for (int j = 0; j < LB; j++) {
            const bool v = k0 + j < e && q[j] >= 0;
#pragma unroll
            for (int k = 0; k < K; k++) c[k] = v && cnt == k ? q[j] : c[k];
            cnt += v ? 1 : 0;
        }
    }
    deg = ((e - b) << 8) | (cnt > K ? K + 1 : cnt);
    NbCache r;
#pragma unroll
    for (int k = 0; k < KQ; k++) {
        r.q[k].x = c[4 * k];
        r.q[k].y = c[4 * k + 1];
        r.q[k].z = c[4 * k + 2];
        r.q[k].w = c[4 * k + 3];
    }
    return r;
}

__device__ __forceinline__ void cache_store(PoolSlot &ps, const NbCache &c)
{
#pragma unroll
    for (int k = 0; k < KQ; k++) ((i32x4 *)ps.nb)[k] = c.q[k];
}

__device__ __forceinline__ void list_add(const Sim &s, int32_t i, int32_t nd)
{
    PoolSlot &ps = s.S.pool(i);
    const int32_t pd = ps.deg;
    const int32_t c = pd & 0xFF;
    if (c > K) return;
    if (c < K) ps.nb[c] = nd;
    ps.deg = (pd & ~0xFF) | (c + 1);
}

// returns false if nd was not cached (cannot happen while the caches are consistent)
__device__ __forceinline__ bool list_remove(const Sim &s, int32_t i, int32_t nd)
{
    PoolSlot &ps = s.S.pool(i);
    int32_t v[K];
#pragma unroll
    for (int k = 0; k < KQ; k++) {
        const i32x4 q = ((const i32x4 *)ps.nb)[k];
        v[4 * k] = q.x;
        v[4 * k + 1] = q.y;
        v[4 * k + 2] = q.z;
        v[4 * k + 3] = q.w;
    }
    const int32_t pd = ps.deg;
    const int32_t c = pd & 0xFF;
    if (c > K) return true;
    int32_t at = -1;
#pragma unroll
    for (int k = 0; k < K; k++)
        if (k < c && v[k] == nd) at = k;
    if (at < 0) return false;
    int32_t lastv = v[0];
#pragma unroll
    for (int k = 0; k < K; k++)
        if (k == c - 1) lastv = v[k];
    ps.nb[at] = lastv;
    ps.nb[c - 1] = 0;
    ps.deg = (pd & ~0xFF) | (c - 1);
    return true;
}

// ------------------------------------------- walk workgroup control --

// Control block of the walk heuristics' workgroup in LDS: what the simulating
// wavefront posts for a scan, the shared candidate counter, the count of
// large walks, and each wavefront's best candidate and work counters.
struct WaveBest {
    uint64_t N, da, db;
    int32_t id, slot, have, pad;
    int64_t nbr, adj, scored;
};
struct WalkCtl {
    int32_t cmd, sim, end, both, use_m, use_s, sample, trace;
    uint32_t ctr, ovf, ctr2, pad;
    int64_t T, evict_no;
    uint64_t min_size, tau, seed;
    WaveBest res[MAX_WALK_WAVES];
};
enum { CMD_WALK = 1, CMD_DONE = 2 };
constexpr int CTL_NODES = (int)((sizeof(WalkCtl) + sizeof(UfNode) - 1) / sizeof(UfNode));

// Order this wavefront's LDS and global accesses (what a workgroup barrier
// gives a one-wave workgroup) without waiting for the other wavefronts.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
}

// wavefronts per workgroup that hold simulations of their own (each with its
// own LDS pool and node arrays): the exact h_DTR^eq kernel's four, else one
__host__ __device__ constexpr int lds_waves(int hc) { return hc == HC_EQ ? EQ_WAVES : 1; }

// the simulating wavefront's synchronization: wavefront-local where its
// workgroup holds other wavefronts (walk heuristics, h_DTR^eq), a workgroup
// barrier otherwise (one-wave workgroups)
template <int HC>
__device__ __forceinline__ void slot_sync()
{
    if constexpr (cls(HC) == HC_WALK || lds_waves(HC) > 1) wave_sync();
    else __syncthreads();
}


// ---------------------------------------------------------------- pool --

// Squeeze tombstones out of the pool (order preserved; positions updated).
template <int HC>
__device__ __forceinline__ void pool_compact(Sim &s)
{
    const int32_t lane = s.lane;
    int32_t kept = 0;
#ifdef DTR_PROFILE
    s.prof_pool_compact++;
#endif
    slot_sync<HC>();
    for (int32_t base = 0; base < s.pool_end; base += WAVE) {
        const int32_t i = base + lane;
        const i32x4 *P = (const i32x4 *)&s.S.pool(i < s.pool_end ? i : 0);
        const i32x4 q0 = P[0], q1 = P[1];
        i32x4 qc[KQ];
#pragma unroll
        for (int k = 0; k < KQ; k++) qc[k] = cls(HC) != HC_SIMPLE ? P[2 + k] : 0;
        const int32_t x = i < s.pool_end ? q0.x : -1;
        const bool keep = x >= 0;
        const uint64_t m = __ballot(keep);
        slot_sync<HC>();
        if (keep) {
            const int32_t j = kept + lane_rank(m);
            i32x4 *Q = (i32x4 *)&s.S.pool(j);
            Q[0] = q0;
            Q[1] = q1;
            if (cls(HC) != HC_SIMPLE)
#pragma unroll
                for (int k = 0; k < KQ; k++) Q[2 + k] = qc[k];
            s.S.tst[x] = ts_make(S_RESIDENT, (uint32_t)j, 0);
        }
        kept += __popcll(m);
        slot_sync<HC>();
    }
    s.pool_end = kept;
}

// Every lane with `want` appends tensor x (resident, unlocked) with last
// access `last`; returns its slot (or -1).  The caller stores x's new state.
// `known`: x's record when the caller holds it already (uniform x).
template <int HC>
__device__ __forceinline__ int32_t pool_append(Sim &s, bool want, int32_t x, int64_t last, const TRec *known = nullptr)
{
    const uint64_t m = __ballot(want);
    if (!m) return -1;
    const int32_t cnt = __popcll(m);
    if (s.pool_end + cnt > s.S.pcap) {
        pool_compact<HC>(s);
        if (s.pool_end + cnt > s.S.pcap) { set_status(s, ST_CAPACITY); return -1; }
    }
    int32_t i = -1;
    if (want) {
        i = s.pool_end + lane_rank(m);
        // the record and the first neighbours are one 64-byte element
        const GAS i32x4 *px = (const GAS i32x4 *)&s.t.rec[x];
        i32x4 hd[2];
        if (cls(HC) != HC_SIMPLE) {
            hd[0] = px[2];
            hd[1] = px[3];
        }
        const TRec r = known ? *known : rec_v(s, x);
        // walk heuristics: the low byte holds the parent count (255: read the record)
        int32_t deg = (r.adj_e - r.adj_b) << 8 | (cls(HC) == HC_WALK ? min(r.in_e - r.in_b, 255) : 0);
        NbCache nb;
        if (cls(HC) == HC_EQ) nb = list_build(s, r.adj_b, r.adj_e, deg, hd);
        i32x4 q0, q1;
        q0.x = x;
        q0.y = deg;
        q0.z = (int32_t)(uint32_t)(uint64_t)last;
        q0.w = (int32_t)(uint32_t)((uint64_t)last >> 32);
        q1.x = (int32_t)(uint32_t)(uint64_t)r.size;
        q1.y = (int32_t)(uint32_t)((uint64_t)r.size >> 32);
        q1.z = r.c0;
        q1.w = r.adj_b;
        i32x4 *Q = (i32x4 *)&s.S.pool(i);
        Q[0] = q0;
        Q[1] = q1;
        if (cls(HC) == HC_EQ) cache_store(s.S.pool(i), nb);
        if (cls(HC) == HC_WALK) {
            // the first neighbours, so that a walk starts from the slot alone
            Q[2] = hd[0];
            Q[3] = hd[1];
        }
    }
    s.pool_end += cnt;
    s.pool_live += cnt;
    return i;
}

// ---------------------------------------------------------- union-find --

// Union-find node access: straight from LDS while every node id is below
// UF_LDS, else through the hybrid store (flat pointers).
struct LdsNodes {
    LAS UfNode *p;
    __device__ __forceinline__ int32_t parent(int32_t i) const { return p[i].parent; }
    __device__ __forceinline__ int32_t size(int32_t i) const { return p[i].size; }
    __device__ __forceinline__ int64_t cost(int32_t i) const { return p[i].cost; }
    __device__ __forceinline__ void set_parent(int32_t i, int32_t v) const { p[i].parent = v; }
    __device__ __forceinline__ void set_size(int32_t i, int32_t v) const { p[i].size = v; }
    __device__ __forceinline__ void set_cost(int32_t i, int64_t v) const { p[i].cost = v; }
};
struct AnyNodes {
    NodeStore n;
    __device__ __forceinline__ int32_t parent(int32_t i) const { return n[i].parent; }
    __device__ __forceinline__ int32_t size(int32_t i) const { return n[i].size; }
    __device__ __forceinline__ int64_t cost(int32_t i) const { return n[i].cost; }
    __device__ __forceinline__ void set_parent(int32_t i, int32_t v) const { n[i].parent = v; }
    __device__ __forceinline__ void set_size(int32_t i, int32_t v) const { n[i].size = v; }
    __device__ __forceinline__ void set_cost(int32_t i, int64_t v) const { n[i].cost = v; }
};


template <class NS>
__device__ __forceinline__ int32_t find_in(const NS &N, int32_t x, int32_t limit)
{
    for (int32_t k = 0; k <= limit; k++) {
        const int32_t p = N.parent(x);
        if (p == x) return x;
        x = p;
    }
    return -1;   // not a forest: reported as a capacity error
}

__device__ __forceinline__ int32_t find_ro(const NodeStore &nodes, int32_t x, int32_t limit)
{
    for (int32_t k = 0; k <= limit; k++) {
        const int32_t p = nodes[x].parent;
        if (p == x) return x;
        x = p;
    }
    return -1;   // not a forest: reported as a capacity error
}

// uniform find with path compression (used where one set is touched)
template <class NS>
__device__ __forceinline__ int32_t find_compress(Sim &s, const NS &N, int32_t x)
{
    int32_t root = x;
    for (int32_t k = 0;; k++) {
        const int32_t p = uni(N.parent(root));
        if (p == root) break;
        if (k > s.uf_n) { set_status(s, ST_CAPACITY); return x; }
        root = p;
    }
    while (x != root) {
        const int32_t nx = uni(N.parent(x));
        N.set_parent(x, root);
        x = nx;
    }
    return root;
}

// Rebuild the node pool: one node per distinct set that still holds an
// evicted tensor (sets left with phantom members only are unreachable).
// Membership and running costs are unchanged, so every later score is too;
// the neighbour caches are rebuilt with the new node ids.
__device__ __forceinline__ void uf_compact(Sim &s)
{
    const int32_t lane = s.lane, n = s.t.n;
    const NodeStore &N = s.S.nodes;
    GAS int32_t *R = s.S.remap;
#ifdef DTR_PROFILE
    s.prof_uf_compact++;
#endif
    wave_sync();
    for (int32_t i = lane; i < s.uf_n; i += WAVE) R[i] = -1;
    wave_sync();
    for (int32_t x = lane; x < n; x += WAVE) {
        const uint64_t w = s.S.tst[x];
        const int32_t v = ts_sw(w);
        if (v >= 0) {
            int32_t r = find_ro(N, v, s.uf_n);
            if (r < 0) r = v;        // cannot happen in a forest; keeps indices in range
            s.S.tst[x] = ts_make(v, (uint32_t)r, ts_locks(w));   // pos is unused while evicted
            R[r] = 0;
        }
    }
    wave_sync();
    int32_t kept = 1;                    // node 0 stays the null node
    for (int32_t base = 0; base < s.uf_n; base += WAVE) {
        const int32_t i = base + lane;
        const bool keep = i > 0 && i < s.uf_n && R[i] == 0;
        const int64_t c = keep ? N[i].cost : 0;
        const uint64_t m = __ballot(keep);
        wave_sync();
        if (keep) {
            const int32_t ni = kept + lane_rank(m);
            R[i] = ni;
            UfNode nd;
            nd.cost = c;
            nd.parent = ni;
            nd.size = 1;
            N[ni] = nd;
        }
        kept += __popcll(m);
        wave_sync();
    }
    for (int32_t x = lane; x < n; x += WAVE) {
        const uint64_t w = s.S.tst[x];
        if (ts_sw(w) >= 0) s.S.tst[x] = ts_make(R[ts_pos(w)], 0, ts_locks(w));
    }
    wave_sync();
    s.uf_n = kept;
    // stay inside LDS while the live sets fit comfortably, else double
    s.uf_limit = kept + 256 <= UF_LDS ? UF_LDS : min(UF_LDS + s.S.ucap, 2 * kept + 256);
    for (int32_t i = lane; i < s.pool_end; i += WAVE) {
        PoolSlot &ps = s.S.pool(i);
        const int32_t x = ps.id;
        if (x >= 0) {
            const TRec r = rec_v(s, x);
            int32_t deg;
            cache_store(ps, list_build(s, r.adj_b, r.adj_e, deg));
            ps.deg = deg;
        }
    }
    wave_sync();
}

// ------------------------------------------------------------ eviction --

// v's fresh node nd (cost c0(v)) joins the sets of all v's evicted neighbours
// (found in parallel, merged under the largest; ties: the earliest), and every
// neighbour waiting in the pool caches nd.
template <class NS>
__device__ __forceinline__ bool evict_merge(Sim &s, const NS &N, int32_t nd, const TRec &rv, int32_t head)
{
    int32_t R = nd;               // current root of v's set
    int64_t Rcost = rv.c0;
    int32_t Rsize = 1;
    if (s.lane == 0) {
        N.set_cost(nd, rv.c0);
        N.set_parent(nd, nd);
        N.set_size(nd, 1);
    }
    bool bad = false;
    for (int32_t k0 = rv.adj_b; k0 < rv.adj_e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        int32_t q = -1, r = -1;
        if (k < rv.adj_e) {
            const uint64_t w = s.S.tst[k0 == rv.adj_b && s.lane < NB_HEAD ? head : gld(s.t.adj + k)];
            q = ts_sw(w);
            if (ts_in_pool(w)) list_add(s, (int32_t)ts_pos(w), nd);
            if (q >= 0) {
                r = find_in(N, q, s.uf_n);
                if (r < 0) { bad = true; r = -1; q = -1; }
            }
        }
        // first lane holding each distinct root contributes it
        bool first = r >= 0;
        uint64_t m = __ballot(r >= 0);
        while (m) {
            const int32_t j = __ffsll((long long)m) - 1;
            m &= m - 1;
            const int32_t rj = __builtin_amdgcn_readlane(r, j);
            if (r == rj && s.lane > j) first = false;
        }
        if (!first || r == R) r = -1;
        int64_t rc = 0;
        int32_t rs = 0;
        if (r >= 0) {
            rc = N.cost(r);
            rs = N.size(r);
        }
        // merge every distinct root into the largest (ties: the earliest)
        uint64_t mr = __ballot(r >= 0);
        int32_t big = R, bigsize = Rsize;
        int64_t sumc = Rcost;
        int32_t sums = Rsize;
        uint64_t mm = mr;
        while (mm) {
            const int32_t j = __ffsll((long long)mm) - 1;
            mm &= mm - 1;
            const int32_t rj = __builtin_amdgcn_readlane(r, j);
            const int32_t sj = __builtin_amdgcn_readlane(rs, j);
            sumc += (int64_t)readlane64((uint64_t)rc, j);
            sums += sj;
            if (sj > bigsize) { big = rj; bigsize = sj; }
        }
        if (mr) {
            if (r >= 0 && r != big) N.set_parent(r, big);
            if (q >= 0 && q != big) N.set_parent(q, big);     // compress the neighbour's path
            if (s.lane == 0 && R != big) N.set_parent(R, big);
            R = big;
            Rcost = sumc;
            Rsize = sums;
        }
    }
    if (__ballot(bad)) { set_status(s, ST_CAPACITY); return false; }
    if (s.lane == 0) {
        N.set_cost(R, Rcost);
        N.set_size(R, Rsize);
        if (nd != R) N.set_parent(nd, R);
    }
    return true;
}

// Evict v (resident, unlocked, in pool slot `slot`).  Under h_DTR^eq, v gets a
// fresh node holding c0(v), which is merged with the sets of all its evicted
// neighbours (found in parallel, merged under the largest), and every
// neighbour waiting in the pool caches the new node.
template <int HC>
__device__ __forceinline__ bool evict(Sim &s, int32_t v, int32_t slot, bool eager)
{
    // size, c0 and neighbour range come from v's pool slot (LDS for the pool
    // head), not from the static record; the first neighbours from the
    // fixed-stride table, read at once
    const int32_t head = cls(HC) == HC_EQ ? gld(s.t.rec[v].nb + (s.lane & (NB_HEAD - 1))) : 0;
    TRec rv;
    {
        const i32x4 *P = (const i32x4 *)&s.S.pool(slot);
        const i32x4 q0 = P[0], q1 = P[1];
        rv.size = uni64((int64_t)(((uint64_t)(uint32_t)q1.y << 32) | (uint32_t)q1.x));
        rv.c0 = uni(q1.z);
        rv.adj_b = uni(q1.w);
        rv.adj_e = rv.adj_b + uni(q0.y >> 8);
    }
    s.S.pool(slot).id = -1;
    s.pool_live--;
    s.mem -= rv.size;
    if (eager) s.eager++;
    else s.evictions++;
    if (cls(HC) != HC_EQ) {
        s.S.tst[v] = ts_make(0, 0, 0);
        return true;
    }
    if (s.uf_n >= s.uf_limit) {
        uf_compact(s);
        if (s.uf_n >= UF_LDS + s.S.ucap) { set_status(s, ST_CAPACITY); return false; }
    }
    const int32_t nd = s.uf_n++;
    bool ok;
    if (s.uf_n <= UF_LDS) {
        LdsNodes NL;
        NL.p = s.S.nodes.lds_l;
        ok = evict_merge(s, NL, nd, rv, head);
    } else {
        AnyNodes NA;
        NA.n = s.S.nodes;
        ok = evict_merge(s, NA, nd, rv, head);
    }
    if (!ok) return false;
    s.S.tst[v] = ts_make(nd, 0, 0);
    return true;
}

// ---------------------------------------------------------------- scan --

// Set roots of the neighbours k0 .. k0+LB-1 (below e) of a candidate: r[j] is
// the root of neighbour k0+j if it is evicted, else -1.  All neighbour and
// state reads are issued together; the finds then advance in lockstep, with
// the first hop compressed (every lane writes the same root).  Returns the
// number of evicted neighbours in the chunk; `bad` is set on a broken forest.
template <class NS>
__device__ __forceinline__ int32_t chunk_roots(const Sim &s, const NS &N, int32_t k0, int32_t e, int32_t (&r)[LB],
                                               bool &bad)
{
    int32_t w[LB], q[LB];
#pragma unroll
    for (int j = 0; j < LB; j++) w[j] = gld(s.t.adj + (k0 + j < e ? k0 + j : k0));
#pragma unroll
    for (int j = 0; j < LB; j++) q[j] = ts_sw(s.S.tst[w[j]]);
    int32_t cnt = 0;
#pragma unroll
    for (int j = 0; j < LB; j++) {
        const bool v = k0 + j < e && q[j] >= 0;
        q[j] = v ? q[j] : 0;            // node 0: the null node, its own root
        r[j] = q[j];
        cnt += v ? 1 : 0;
    }
    for (int32_t it = 0;; it++) {
        int32_t p[LB];
        bool more = false;
#pragma unroll
        for (int j = 0; j < LB; j++) {
            p[j] = N.parent(r[j]);
            more |= p[j] != r[j];
        }
        if (!more) break;
        if (it > s.uf_n) { bad = true; break; }
#pragma unroll
        for (int j = 0; j < LB; j++) r[j] = p[j];
    }
#pragma unroll
    for (int j = 0; j < LB; j++) {
        if (q[j] != 0 && r[j] != q[j]) N.set_parent(q[j], r[j]);
        r[j] = q[j] != 0 ? r[j] : -1;
    }
    return cnt;
}

// Neighbourhood cost under h_DTR^eq from the full adjacency [b, e) (used when
// the candidate's cache overflowed or a cached node sits deep in its set):
// summed running costs of the distinct sets of its evicted neighbours.  A
// set counts at its first neighbour; chunks after the first compare against
// the roots of the chunks before them.
template <class NS>
__device__ __forceinline__ int64_t eq_cost_full(const Sim &s, const NS &N, int32_t b, int32_t e, int64_t &ev_count,
                                                bool &bad)
{
    int64_t sum = 0, cnt = 0;
    for (int32_t k0 = b; k0 < e; k0 += LB) {
        int32_t r[LB];
        cnt += chunk_roots(s, N, k0, e, r, bad);
        bool keep[LB];
#pragma unroll
        for (int j = 0; j < LB; j++) {
            keep[j] = r[j] >= 0;
#pragma unroll
            for (int i = 0; i < j; i++) keep[j] = keep[j] && r[i] != r[j];
        }
        for (int32_t p0 = b; p0 < k0; p0 += LB) {
            int32_t rp[LB];
            chunk_roots(s, N, p0, e, rp, bad);
#pragma unroll
            for (int j = 0; j < LB; j++)
#pragma unroll
                for (int i = 0; i < LB; i++) keep[j] = keep[j] && rp[i] != r[j];
        }
#pragma unroll
        for (int j = 0; j < LB; j++) sum += keep[j] ? N.cost(r[j]) : 0;
    }
    ev_count = cnt;
    return sum;
}

// Scores are N / (da * db) with N < 2^64 and da * db < 2^76.  A float
// estimate decides every comparison whose two estimates differ by more than a
// factor 1 -+ 2^-16; the rest (near ties, exact ties, 0/0) are decided
// exactly by 128-bit cross-multiplication, so the outcome is always that of
// the exact comparison.  Error of the estimate: each u64f conversion rounds
// twice (the high and low 32-bit halves, then the fused sum), under
// (1 + 2^-24)^2 - 1 < 2^-22.9; the product da * db adds one rounding
// (2^-24), v_rcp_f32 at most 1 ulp (2^-23) and the final product one
// rounding (2^-24): in all below 3 * 2^-22.9 + 2^-23 + 2 * 2^-24 < 2^-20.4.
// Two estimates within the margin can therefore never be ordered wrongly by
// the float test: (1 - 2^-16) (1 + 2^-24) (1 + 2^-20.4)^2 < 1.
constexpr float FILTER_LO = 1.0f - 0x1p-16f;
constexpr float FILTER_HI = 1.0f + 0x1p-16f;

__device__ __forceinline__ float u64f(uint64_t x)
{
    return fmaf((float)(uint32_t)(x >> 32), 4294967296.0f, (float)(uint32_t)x);
}

__device__ __forceinline__ float score_est(uint64_t N, uint64_t da, uint64_t db)
{
    return u64f(N) * __builtin_amdgcn_rcpf(u64f(da) * u64f(db));   // 0 -> inf, 0/0 -> NaN
}

__device__ __forceinline__ bool better_exact(uint64_t na, uint64_t daa, uint64_t dba, int32_t ia, uint64_t nb,
                                             uint64_t dab, uint64_t dbb, int32_t ib)
{
    return better(na, (u128)daa * dba, ia, nb, (u128)dab * dbb, ib);
}

struct Best {
    float sc, lo, hi;    // estimated score of the best and its decision bounds
    uint64_t N, da, db;
    int32_t id, slot, have;
};

// keep the candidate if valid and better than the current best
__device__ __forceinline__ void take(Best &b, bool valid, float sc, uint64_t N, uint64_t da, uint64_t db, int32_t id,
                                     int32_t slot)
{
    const bool dec_better = sc < b.lo;
    const bool dec_worse = sc > b.hi;
    bool t = valid && (!b.have || dec_better);
    const bool close = valid && b.have && !dec_better && !dec_worse;
    if (__ballot(close)) {
        if (close) t = better_exact(N, da, db, id, b.N, b.da, b.db, b.id);
    }
    b.sc = t ? sc : b.sc;
    b.lo = t ? sc * FILTER_LO : b.lo;
    b.hi = t ? sc * FILTER_HI : b.hi;
    b.N = t ? N : b.N;
    b.da = t ? da : b.da;
    b.db = t ? db : b.db;
    b.id = t ? id : b.id;
    b.slot = t ? slot : b.slot;
    b.have = t ? 1 : b.have;
}

// Which candidates an eviction decision searches (the prototype's search
// approximations, Appendix E): those of size >= min_size (size at least 1% of
// the pool's mean: 100 size n0 >= sum of sizes, i.e. size >= ceil(sum / (100
// n0)); 0 without the flag) and, with `sample`, whose sampling draw is below
// tau (probability ceil(sqrt(n0))/n0).
struct Filter {
    bool sample;
    uint64_t min_size, tau;
};

__device__ __forceinline__ uint64_t sample_draw(const Sim &s, int32_t x)
{
    const uint64_t key = ((uint64_t)s.evict_no << 32) + (uint64_t)(uint32_t)x;
    return mix64((s.seed ^ 0xD6E8FEB86659FD93ull) + 0x9E3779B97F4A7C15ull * key);
}

// filter of the first search pass; `sample` stays off when it would keep
// every candidate (ceil(sqrt(n0)) >= n0)
template <int HC>
__device__ __forceinline__ Filter make_filter(Sim &s)
{
    Filter F;
    const uint32_t n0 = (uint32_t)s.pool_live;
    F.min_size = 0;
    if (s.search & SEARCH_IGNORE_SMALL) {
        uint64_t sum = 0;
        for (int32_t i = s.lane; i < s.pool_end; i += WAVE) {
            const i32x4 *P = (const i32x4 *)&s.S.pool(i);
            const i32x4 q0 = P[0], q1 = P[1];
            if (q0.x >= 0) sum += ((uint64_t)(uint32_t)q1.y << 32) | (uint32_t)q1.x;
        }
        for (int off = WAVE / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, WAVE);
        sum = (uint64_t)uni64((int64_t)sum);
        const uint64_t d = 100 * (uint64_t)n0;
        F.min_size = (sum + d - 1) / d;
    }
    F.sample = false;
    F.tau = 0;
    if (s.search & SEARCH_SAMPLE) {
        uint32_t k = (uint32_t)sqrtf((float)n0);          // then corrected to ceil(sqrt(n0))
        while (k * k < n0) k++;
        while (k > 0 && (k - 1) * (k - 1) >= n0) k--;
        if (k < n0) {
            // tau = floor(k 2^64 / n0) by long division in two 32-bit digits
            const uint64_t a = (uint64_t)k << 32;
            const uint64_t q1 = a / n0, r1 = a % n0;
            const uint64_t q2 = (r1 << 32) / n0;
            F.tau = (q1 << 32) + q2;
            F.sample = true;
        }
    }
    return F;
}

// Score every searched pool entry; return the victim (uniform) and its slot,
// or -1; `scored` receives the number of candidates scored.
// Sum of the set costs behind the first KK cached nodes of a candidate (nodes
// in LDS): each node's parent is the set root unless the node is more than one
// merge away (then `deep` is set and the caller recounts); equal roots count
// once.
template <int KK>
__device__ __forceinline__ int64_t cached_sum(const LAS UfNode *NL, const int32_t (&nb)[K], bool &deep)
{
    const LAS i32x4 *NQ = (const LAS i32x4 *)NL;    // {cost lo, cost hi, parent, size}
    int32_t r[KK];
    int64_t cost[KK];
#pragma unroll
    for (int k = 0; k < KK; k++) r[k] = NL[nb[k]].parent;
#pragma unroll
    for (int k = 0; k < KK; k++) {
        const i32x4 n2 = NQ[r[k]];
        cost[k] = (int64_t)(((uint64_t)(uint32_t)n2.y << 32) | (uint32_t)n2.x);
        deep |= n2.z != r[k];
    }
    int64_t t = 0;
#pragma unroll
    for (int k = 0; k < KK; k++) {
        bool dup = false;
#pragma unroll
        for (int j = 0; j < k; j++) dup |= r[j] == r[k];
        t += dup ? 0 : cost[k];
    }
    return t;
}

// ------------------------------------------------------------- e* walks --

// What a walk scan needs to know, identical in every lane and wavefront.
struct WalkParams {
    int32_t end, both, use_m, use_s, sample;
    int64_t T, evict_no;
    uint64_t min_size, tau, seed;
};

// the search approximations' sampling draw of candidate x (Appendix E)
__device__ __forceinline__ uint64_t sample_draw_at(uint64_t seed, int64_t evict_no, int32_t x)
{
    const uint64_t key = ((uint64_t)evict_no << 32) + (uint64_t)(uint32_t)x;
    return mix64((seed ^ 0xD6E8FEB86659FD93ull) + 0x9E3779B97F4A7C15ull * key);
}

// The evicted neighbourhood walks of one wavefront, one candidate per lane.
// Each lane takes the next pool slot (from the workgroup's LDS counter when
// wavefronts share the scan) as soon as its previous walk has ended, and
// expands one tensor per iteration.  The candidate x comes from its pool slot
// alone (which holds its first neighbours and parent count): its evicted
// parents start its ancestors (e_R) and, for e*, its evicted children its
// descendants.  Then each queued member: its record element brings its cost
// c0 and first neighbours; an ancestor-side member follows its parents (the
// first neighbours), a descendant-side member its children (read from the
// adjacency list).  The two sides are disjoint in a DAG, so one visited flag
// per tensor serves both: a byte per tensor and lane, so that marks need no
// read-modify-write.  Up to NC neighbours are checked per iteration, their
// reads issued together; a tensor with more relevant neighbours keeps its
// cursor for the next iteration.  A member is marked and queued at once, so
// the queue lists exactly the marked tensors and the flags are cleared from
// it after the walk.  A walk ends, and is scored, in the iteration that
// leaves its queue empty.  A walk that would outgrow the lane's queue is
// abandoned (cleared) and its slot listed: those are walked afterwards by
// whole wavefronts.
template <int HC>
__device__ void walk_lanes(const TraceDev &t, const Slot &S, GAS uint64_t *tst, const WalkParams &P,
                           int32_t lane, int32_t lid, LAS uint32_t *ctr, LAS uint32_t *novf, Best &best,
                           int64_t &nbr, int64_t &adj, int64_t &nscored)
{
    constexpr int NC = 8;                 // neighbours checked per iteration
    GAS uint8_t *vis = S.visb + (size_t)lid * (size_t)S.vis_bytes;
    GAS int32_t *q = S.wq + (size_t)lid * (size_t)S.wq_cap;
    const GAS int32_t *sw = (const GAS int32_t *)tst;     // low words of the state words
    const int32_t cap = S.wq_cap;
    int32_t next = 0;                     // next pool slot (one wavefront alone)
    bool drained = false;
    int32_t x = -1, slot = 0, deg = 0, head = 0, tail = 0;
    int64_t sum = 0, c0x = 0, size = 0, last = 0;
    // the tensor being expanded: neighbour cursor k over [k, ke) of its
    // adjacency (base ab, np parents first), side of the members it finds
    // (-1: the candidate), and its first neighbours (from the pool slot or
    // the record element), used while the cursor is at 0
    int32_t k = 0, ke = 0, ab = 0, np = 0, sd = 0;
    int32_t nb[NB_HEAD];
#pragma unroll
    for (int c = 0; c < NB_HEAD; c++) nb[c] = 0;
    for (;;) {
        const bool idle = x < 0;
        const uint64_t mi = __ballot(idle);
        uint32_t i = 0xffffffffu;
        if (mi && !drained) {
            uint32_t b;
            if (ctr) {
                const int32_t first = __ffsll((long long)mi) - 1;
                uint32_t got = 0;
                if (lane == first) got = atomicAdd((uint32_t *)ctr, (uint32_t)__popcll(mi));
                b = (uint32_t)__builtin_amdgcn_readlane((int32_t)got, first);
            } else {
                b = (uint32_t)next;
                next += __popcll(mi);
            }
            if (b + (uint32_t)__popcll(mi) >= (uint32_t)P.end) drained = true;
            if (idle) i = b + (uint32_t)lane_rank(mi);
        } else if (!__ballot(x >= 0)) {
            break;
        }
        if (i < (uint32_t)P.end) {
            i32x4 q0, q1, h0, h1;
            if (i < (uint32_t)POOL_LDS) {
                const LAS i32x4 *PS = (const LAS i32x4 *)S.lpool_l + PQL * i;
                q0 = PS[0]; q1 = PS[1]; h0 = PS[2]; h1 = PS[3];
            } else {
                const GAS i32x4 *PS = (const GAS i32x4 *)S.gpool + PQ * (size_t)i;
                q0 = PS[0]; q1 = PS[1]; h0 = PS[2]; h1 = PS[3];
            }
            bool ok = q0.x >= 0;
            const int64_t sz = (int64_t)(((uint64_t)(uint32_t)q1.y << 32) | (uint32_t)q1.x);
            if (approx(HC)) {
                ok = ok && (uint64_t)sz >= P.min_size;
                if (P.sample) ok = ok && sample_draw_at(P.seed, P.evict_no, q0.x) < P.tau;
            }
            if (ok) {
                x = q0.x;
                slot = (int32_t)i;
                deg = q0.y >> 8;
                last = (int64_t)(((uint64_t)(uint32_t)q0.w << 32) | (uint32_t)q0.z);
                size = sz;
                c0x = (int64_t)q1.z;
                head = tail = 0;
                sum = 0;
                np = q0.y & 0xFF;
                if (np == 255) {                // 255 or more parents: the record has the count
                    const TRec r = rec_v_t(t, x);
                    np = r.in_e - r.in_b;
                }
                ab = q1.w;
                k = 0;
                ke = P.both ? deg : np;
                sd = -1;
                nb[0] = h0.x; nb[1] = h0.y; nb[2] = h0.z; nb[3] = h0.w;
                nb[4] = h1.x; nb[5] = h1.y; nb[6] = h1.z; nb[7] = h1.w;
            }
        } else if (x >= 0 && k >= ke) {
            // the next queued member
            const int32_t e = q[head++];
            const int32_t u = e & 0x7fffffff;
            const GAS i32x4 *R = (const GAS i32x4 *)&t.rec[u];
            const i32x4 r0 = R[0], r1 = R[1], n0 = R[2], n1 = R[3];
            sum += (int64_t)r0.z;
            np = r1.y - r1.x;
            ab = r1.z;
            sd = (int32_t)((uint32_t)e >> 31);
            k = sd == 0 ? 0 : np;
            ke = sd == 0 ? np : r1.w - r1.z;
            nb[0] = n0.x; nb[1] = n0.y; nb[2] = n0.z; nb[3] = n0.w;
            nb[4] = n1.x; nb[5] = n1.y; nb[6] = n1.z; nb[7] = n1.w;
        }
        bool over = false;
        if (x >= 0 && k < ke) {
            // up to NC neighbours from the cursor: the first NB_HEAD from the
            // registers when the cursor is at 0, the rest from the adjacency
            // list; a lane reads only the neighbours in its range
            int32_t v[NC], st[NC];
            uint8_t seen[NC];
#pragma unroll
            for (int j = 0; j < NC; j++) {
                v[j] = (k == 0 && j < NB_HEAD) ? nb[j] : 0;
                if (k + j < ke && !(k == 0 && j < NB_HEAD)) v[j] = gld(t.adj + ab + k + j);
            }
#pragma unroll
            for (int j = 0; j < NC; j++) {
                st[j] = -1;
                seen[j] = 1;
                if (k + j < ke) {
                    st[j] = sw[2 * (size_t)v[j]];
                    seen[j] = vis[v[j]];
                }
            }
#pragma unroll
            for (int j = 0; j < NC; j++) {
                if (st[j] >= 0 && !seen[j]) {
                    if (tail >= cap) {
                        over = true;
                    } else {
                        vis[v[j]] = 1;
                        const int32_t s2 = sd >= 0 ? sd : (k + j < np ? 0 : 1);
                        q[tail++] = v[j] | (s2 << 31);
                    }
                }
            }
            k += NC;
        }
        // the walk ends with the expansion that leaves nothing to expand
        const bool fin = x >= 0 && !over && k >= ke && head == tail;
        if (__ballot(fin)) {
            const uint64_t N = (uint64_t)(c0x + sum);
            const uint64_t DA = P.use_m ? (uint64_t)size : 1;
            const uint64_t DB = P.use_s ? (uint64_t)(P.T - last) : 1;
            take(best, fin, fin ? score_est(N, DA, DB) : 0.0f, N, DA, DB, x, slot);
        }
        if (over) {
            // listed for a whole-wavefront walk (its members are recounted there)
            const uint32_t kk = atomicAdd((uint32_t *)novf, 1u);
            S.ovf[kk] = slot;
        }
        if (fin) {
            nbr += tail;
            adj += deg;
            nscored++;
        }
        if (fin || over) {
            // every set flag of the lane belongs to this walk; entries read 8 at a time
            for (int32_t j0 = 0; j0 < tail; j0 += 8) {
                int32_t e[8];
#pragma unroll
                for (int j = 0; j < 8; j++) e[j] = q[min(j0 + j, tail - 1)];
#pragma unroll
                for (int j = 0; j < 8; j++) vis[e[j] & 0x7fffffff] = 0;
            }
            x = -1;
            k = ke = 0;
        }
    }
}

// A whole wavefront walks the evicted neighbourhood of candidate x (uniform)
// with its own bitmap bv and queue bq, a level of up to 64 queued tensors at
// a time: each lane expands one (its record element brings c0 and the first
// neighbours), claims evicted neighbours with an atomic OR on the bitmap, and
// claimed ones are appended in lane order.  Returns the summed c0 of the
// members (uniform); *count gets their number.
__device__ int64_t walk_wave(const TraceDev &t, GAS uint64_t *tst, GAS uint32_t *bv, GAS int32_t *bq, int32_t x,
                             bool both, int32_t lane, int64_t *count)
{
    constexpr int WB = 8;
    int32_t tail = 0;
    int64_t sum = 0;
    // lane's tensor u (or -1) and the side of the members it finds (-1: the
    // candidate, parents to side 0 and children to side 1)
    auto expand = [&](int32_t u, int32_t side) {
        int32_t kb = 0, ke = 0, np = 0, ab = 0;
        int32_t nb[NB_HEAD];
#pragma unroll
        for (int c = 0; c < NB_HEAD; c++) nb[c] = 0;
        if (u >= 0) {
            const GAS i32x4 *R = (const GAS i32x4 *)&t.rec[u];
            const i32x4 r0 = R[0], r1 = R[1], n0 = R[2], n1 = R[3];
            if (side >= 0) sum += (int64_t)r0.z;
            np = r1.y - r1.x;
            ab = r1.z;
            const int32_t dg = r1.w - r1.z;
            kb = side == 1 ? np : 0;
            ke = side < 0 ? (both ? dg : np) : (side == 0 ? np : dg);
            nb[0] = n0.x; nb[1] = n0.y; nb[2] = n0.z; nb[3] = n0.w;
            nb[4] = n1.x; nb[5] = n1.y; nb[6] = n1.z; nb[7] = n1.w;
        }
        for (int32_t c0 = 0; __ballot(kb + c0 < ke); c0 += WB) {
            int32_t v[WB];
            bool claim[WB];
            uint64_t w[WB];
#pragma unroll
            for (int j = 0; j < WB; j++) {
                const int32_t kc = min(kb + c0 + j, max(ke - 1, 0));
                int32_t id = nb[0];
#pragma unroll
                for (int c = 1; c < NB_HEAD; c++) id = kc == c ? nb[c] : id;
                v[j] = kc < NB_HEAD ? id : gld(t.adj + ab + kc);
            }
#pragma unroll
            for (int j = 0; j < WB; j++) w[j] = tst[v[j]];
#pragma unroll
            for (int j = 0; j < WB; j++) {
                claim[j] = false;
                if (kb + c0 + j < ke && ts_sw(w[j]) >= 0) {
                    const uint32_t bit = 1u << (v[j] & 31);
                    claim[j] = !(atomicOr((uint32_t *)(bv + (v[j] >> 5)), bit) & bit);
                }
            }
#pragma unroll
            for (int j = 0; j < WB; j++) {
                const uint64_t m = __ballot(claim[j]);
                if (claim[j]) {
                    const int32_t s2 = side >= 0 ? side : (kb + c0 + j < np ? 0 : 1);
                    bq[tail + lane_rank(m)] = v[j] | (s2 << 31);
                }
                tail += __popcll(m);
            }
        }
    };
    expand(lane == 0 ? x : -1, -1);
    wave_sync();
    for (int32_t head = 0; head < tail;) {
        const int32_t hi = min(tail, head + WAVE);
        int32_t u = -1, side = 0;
        if (head + lane < hi) {
            const int32_t e = bq[head + lane];
            u = e & 0x7fffffff;
            side = (int32_t)((uint32_t)e >> 31);
        }
        head = hi;
        expand(u, side);
        wave_sync();
    }
    for (int32_t j = lane; j < tail; j += WAVE) bv[(bq[j] & 0x7fffffff) >> 5] = 0u;
    wave_sync();
    for (int off = WAVE / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, WAVE);
    *count = tail;
    return uni64(sum);
}

// The listed walks, each by a whole wavefront: wavefronts take them from the
// shared counter ctr2 (this wavefront alone when ctr2 is null) and keep the
// best in `best` (lane 0 takes each result).
template <int HC>
__device__ void walk_listed(const TraceDev &t, const Slot &S, GAS uint64_t *tst, const WalkParams &P, int32_t lane,
                            int32_t wave, int32_t n_ovf, LAS uint32_t *ctr2, Best &best, int64_t &nbr,
                            int64_t &adj, int64_t &nscored)
{
    GAS uint32_t *bv = S.bigvis + (size_t)wave * (size_t)S.vis_words;
    GAS int32_t *bq = S.bigq + (size_t)wave * (size_t)(S.n_max + 1);
    for (int32_t own = 0;;) {
        int32_t k;
        if (ctr2) {
            uint32_t got = 0;
            if (lane == 0) got = atomicAdd((uint32_t *)ctr2, 1u);
            k = uni((int32_t)got);
        } else {
            k = own++;
        }
        if (k >= n_ovf) break;
        const int32_t sl = uni(gld(S.ovf + k));
        const i32x4 *PS = (const i32x4 *)&S.pool(sl);
        const i32x4 q0 = PS[0], q1 = PS[1];
        const int32_t x = uni(q0.x);
        const int64_t last = uni64((int64_t)(((uint64_t)(uint32_t)q0.w << 32) | (uint32_t)q0.z));
        const int64_t size = uni64((int64_t)(((uint64_t)(uint32_t)q1.y << 32) | (uint32_t)q1.x));
        const int64_t c0x = (int64_t)uni(q1.z);
        int64_t cnt = 0;
        const int64_t sum = walk_wave(t, tst, bv, bq, x, P.both, lane, &cnt);
        const uint64_t N = (uint64_t)(c0x + sum);
        const uint64_t DA = P.use_m ? (uint64_t)size : 1;
        const uint64_t DB = P.use_s ? (uint64_t)(P.T - last) : 1;
        const bool me = lane == 0;
        take(best, me, score_est(N, DA, DB), N, DA, DB, x, sl);
        if (me) {
            nbr += cnt;
            adj += uni(q0.y >> 8);
            nscored++;
        }
    }
}

// the wavefront's best (exact lexicographic minimum of score and id over its
// lanes), uniform
__device__ WaveBest wave_best(const Best &best)
{
    WaveBest r;
    float mn = best.have ? best.sc : __builtin_inff();
    for (int off = WAVE / 2; off >= 1; off >>= 1) mn = fminf(mn, __shfl_xor(mn, off, WAVE));
    const float thr = mn * FILTER_HI;
    uint64_t m = __ballot(best.have && !(best.sc > thr));     // NaN estimates stay in
    r.have = m ? 1 : 0;
    r.N = 0;
    r.da = r.db = 1;
    r.id = 0x7fffffff;
    r.slot = -1;
    r.pad = 0;
    r.nbr = r.adj = r.scored = 0;
    while (m) {
        const int32_t j = __ffsll((long long)m) - 1;
        m &= m - 1;
        const uint64_t cN = readlane64(best.N, j), cda = readlane64(best.da, j), cdb = readlane64(best.db, j);
        const int32_t cid = __builtin_amdgcn_readlane(best.id, j), cslot = __builtin_amdgcn_readlane(best.slot, j);
        if (r.slot < 0 || better_exact(cN, cda, cdb, cid, r.N, r.da, r.db, r.id)) {
            r.N = cN;
            r.da = cda;
            r.db = cdb;
            r.id = cid;
            r.slot = cslot;
        }
    }
    return r;
}

__device__ __forceinline__ int64_t wave_sum(int64_t v)
{
    for (int off = WAVE / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, WAVE);
    return uni64(v);
}

// The walk scan of the simulating wavefront.  Helper wavefronts (if any) are
// given the scan's parameters at a workgroup barrier; all wavefronts walk
// candidates lane by lane from the shared counter; after a second barrier
// they take the listed (large) walks one per wavefront; after a third, the
// helpers' bests enter this wavefront's lanes 1.. and their counters are
// added.
template <int HC>
__device__ void walk_scan(Sim &s, const Filter &F, Best &best, int64_t &scored)
{
    WalkParams P;
    P.end = s.pool_end;
    P.both = s.cmode == CM_ESTAR;
    P.use_m = s.use_m;
    P.use_s = s.use_s;
    P.sample = F.sample;
    P.T = s.T;
    P.evict_no = s.evict_no;
    P.min_size = F.min_size;
    P.tau = F.tau;
    P.seed = s.seed;
    LAS WalkCtl *C = s.ctl;
    const bool multi = s.nw > 1;
    if (s.lane == 0) {
        C->ovf = 0;
        C->ctr = 0;
        C->ctr2 = 0;
    }
    if (multi) {
        if (s.lane == 0) {
            C->cmd = CMD_WALK;
            C->trace = s.trace_idx;
            C->end = P.end;
            C->both = P.both;
            C->use_m = P.use_m;
            C->use_s = P.use_s;
            C->sample = P.sample;
            C->T = P.T;
            C->evict_no = P.evict_no;
            C->min_size = P.min_size;
            C->tau = P.tau;
            C->seed = P.seed;
        }
        __syncthreads();
    } else {
        wave_sync();
    }
    int64_t nbr = 0, adj = 0, nscored = 0;
#ifdef DTR_PROFILE
    // walk heuristics: cycles of this wavefront's own walks, of the wait for
    // the helpers, of the whole-wavefront walks, and their number
    const int64_t w1 = (int64_t)__builtin_readcyclecounter();
#endif
    walk_lanes<HC>(s.t, s.S, s.S.tst, P, s.lane, s.lane, multi ? (LAS uint32_t *)&C->ctr : nullptr,
                   (LAS uint32_t *)&C->ovf, best, nbr, adj, nscored);
#ifdef DTR_PROFILE
    const int64_t w2 = (int64_t)__builtin_readcyclecounter();
#endif
    if (multi) __syncthreads();
    else wave_sync();
#ifdef DTR_PROFILE
    const int64_t w3 = (int64_t)__builtin_readcyclecounter();
#endif
    walk_listed<HC>(s.t, s.S, s.S.tst, P, s.lane, 0, uni((int32_t)C->ovf), multi ? (LAS uint32_t *)&C->ctr2 : nullptr,
                    best, nbr, adj, nscored);
#ifdef DTR_PROFILE
    const int64_t w4 = (int64_t)__builtin_readcyclecounter();
    s.prof_rounds += w2 - w1;
    if (s.lane == 0) {
        s.prof_slow += w3 - w2;
        s.prof_global_nodes += w4 - w3;
    }
    s.prof_uf_compact += uni((int32_t)C->ovf);
#endif
    if (multi) {
        __syncthreads();
        // the helpers' bests, one per lane 1..nw-1
        const int32_t w = s.lane < s.nw ? s.lane : 0;
        const bool h = w >= 1 && C->res[w].have;
        const uint64_t N = h ? C->res[w].N : 0, da = h ? C->res[w].da : 1, db = h ? C->res[w].db : 1;
        const int32_t id = h ? C->res[w].id : 0, sl = h ? C->res[w].slot : 0;
        if (__ballot(h)) take(best, h, h ? score_est(N, da, db) : 0.0f, N, da, db, id, sl);
        if (w >= 1) {
            nbr += C->res[w].nbr;
            adj += C->res[w].adj;
            nscored += C->res[w].scored;
        }
    }
    s.nbr += nbr;
    s.adj += adj;
    if (approx(HC)) scored += wave_sum(nscored);
}

// A helper wavefront of a walk heuristic's workgroup: joins the simulating
// wavefront's walk scans (the three workgroup barriers of each) until it is
// released at the end of the simulation.
template <int HC>
__device__ void help_walks(const KernelArgs &a, const Slot &S, int32_t lane, int32_t wave, LAS WalkCtl *C)
{
    for (;;) {
        __syncthreads();
        if (C->cmd == CMD_DONE) break;
        WalkParams P;
        P.end = C->end;
        P.both = C->both;
        P.use_m = C->use_m;
        P.use_s = C->use_s;
        P.sample = C->sample;
        P.T = C->T;
        P.evict_no = C->evict_no;
        P.min_size = C->min_size;
        P.tau = C->tau;
        P.seed = C->seed;
        const TraceDev t = a.traces[C->trace];
        Best best;
        best.sc = best.lo = best.hi = 0.0f;
        best.N = 0;
        best.da = best.db = 1;
        best.id = 0x7fffffff;
        best.slot = -1;
        best.have = 0;
        int64_t nbr = 0, adj = 0, nscored = 0;
        walk_lanes<HC>(t, S, S.tst, P, lane, wave * WAVE + lane, (LAS uint32_t *)&C->ctr, (LAS uint32_t *)&C->ovf,
                       best, nbr, adj, nscored);
        __syncthreads();
        walk_listed<HC>(t, S, S.tst, P, lane, wave, uni((int32_t)C->ovf), (LAS uint32_t *)&C->ctr2, best, nbr, adj,
                        nscored);
        WaveBest r = wave_best(best);
        r.nbr = wave_sum(nbr);
        r.adj = wave_sum(adj);
        r.scored = wave_sum(nscored);
        if (lane == 0) *(WaveBest *)&C->res[wave] = r;
        __syncthreads();
    }
}

// Score the pool rounds of a scan (each WAVE * U entries) into this
// wavefront's per-lane bests; `bad` is set on a broken forest.  Rounds in
// global memory are read one round ahead, so that their latency overlaps the
// scoring of the round before (scans start in LDS).
template <int HC>
__device__ __forceinline__ void scan_rounds(Sim &s, const Filter &F, Best &best, int64_t &scored, bool &bad)
{
    const int32_t end = s.pool_end;
    const int32_t lane = s.lane;
    const int64_t T = s.T;
    const LAS i32x4 *L4 = (const LAS i32x4 *)s.S.lpool_l;
    const GAS i32x4 *G4 = (const GAS i32x4 *)s.S.gpool;
    constexpr int U = Round<HC>::value;
    static_assert(POOL_LDS > 0, "the first round of a scan lies in LDS");
    i32x4 P0[U], P1[U], PC[U][KQ];
    for (int32_t base = 0; base < end; base += WAVE * U) {
        int32_t id[U], pd[U];
        uint32_t slot[U];
        int64_t last[U], size[U], c0[U];
        int32_t ab[U];
        int32_t nb[U][K];
        bool ok[U];
        // level 1: the 16-byte quads of each slot, all issued together, from
        // LDS or global memory (a round never straddles the two)
        i32x4 Q0[U], Q1[U], QC[U][KQ];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int32_t i = base + u * WAVE + lane;
            slot[u] = (uint32_t)(i < end ? i : base);
        }
        if (base < POOL_LDS) {
#pragma unroll
            for (int u = 0; u < U; u++) {
                Q0[u] = L4[PQL * slot[u]];
                Q1[u] = L4[PQL * slot[u] + 1];
#pragma unroll
                for (int k = 0; k < KQ; k++) QC[u][k] = cls(HC) == HC_EQ ? L4[PQL * slot[u] + 2 + k] : 0;
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; u++) {
                Q0[u] = P0[u];
                Q1[u] = P1[u];
#pragma unroll
                for (int k = 0; k < KQ; k++) QC[u][k] = PC[u][k];
            }
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int32_t i = base + u * WAVE + lane;
            const i32x4 q0 = Q0[u], q1 = Q1[u];
            id[u] = i < end ? q0.x : -1;
            pd[u] = q0.y;
            last[u] = (int64_t)(((uint64_t)(uint32_t)q0.w << 32) | (uint32_t)q0.z);
            size[u] = (int64_t)(((uint64_t)(uint32_t)q1.y << 32) | (uint32_t)q1.x);
            c0[u] = (int64_t)q1.z;
            ab[u] = q1.w;
#pragma unroll
            for (int k = 0; k < KQ; k++) {
                nb[u][4 * k] = QC[u][k].x;
                nb[u][4 * k + 1] = QC[u][k].y;
                nb[u][4 * k + 2] = QC[u][k].z;
                nb[u][4 * k + 3] = QC[u][k].w;
            }
            ok[u] = id[u] >= 0;
            if (approx(HC)) {
                ok[u] = ok[u] && (uint64_t)size[u] >= F.min_size;
                if (F.sample) ok[u] = ok[u] && sample_draw(s, id[u]) < F.tau;
            }
        }
        const int32_t nbase = base + WAVE * U;
        if (nbase < end && nbase >= POOL_LDS) {
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int32_t i = nbase + u * WAVE + lane;
                const uint32_t ns = (uint32_t)(i < end ? i : nbase);
                P0[u] = G4[PQ * ns];
                P1[u] = G4[PQ * ns + 1];
#pragma unroll
                for (int k = 0; k < KQ; k++) PC[u][k] = cls(HC) == HC_EQ ? G4[PQ * ns + 2 + k] : 0;
            }
        }
        uint64_t N[U], DA[U], DB[U];
        if (cls(HC) == HC_EQ) {
            const bool lds_nodes = s.uf_n <= UF_LDS;
            // level 2: every cached node (unused entries hold node 0, the null
            // node); level 3: its parent, so nodes one merge away resolve too
            int64_t sum[U], ev[U];
            bool slow[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int32_t c = pd[u] & 0xFF;
                // roots are their own parent, so the node two hops along (n2)
                // is the set root whenever the cached node is at most one
                // merge away from it; its cost is used unconditionally
                bool deep = false;
                // cache entries at or beyond every lane's count hold the null
                // node (cost 0, its own root) and are skipped when the whole
                // wave allows it
                if (lds_nodes) {
                    const LAS UfNode *NL = s.S.nodes.lds_l;
                    if (!__ballot(c > 2)) sum[u] = cached_sum<2>(NL, nb[u], deep);
                    else if (!__ballot(c > 4)) sum[u] = cached_sum<4>(NL, nb[u], deep);
                    else sum[u] = cached_sum<K>(NL, nb[u], deep);
                } else {
                    int32_t r[K];
                    int64_t cost[K];
#pragma unroll
                    for (int k = 0; k < K; k++) r[k] = s.S.nodes[nb[u][k]].parent;
#pragma unroll
                    for (int k = 0; k < K; k++) {
                        const UfNode n2 = s.S.nodes[r[k]];
                        cost[k] = n2.cost;
                        deep |= n2.parent != r[k];
                    }
                    int64_t t = 0;
#pragma unroll
                    for (int k = 0; k < K; k++) {
                        bool dup = false;
#pragma unroll
                        for (int j = 0; j < k; j++) dup |= r[j] == r[k];
                        t += dup ? 0 : cost[k];
                    }
                    sum[u] = t;
                }
                ev[u] = c;
                slow[u] = ok[u] && (c > K || deep);
            }
            // rare: overflowed cache or a merged-away node -- exact recount
            bool any_slow = false;
#pragma unroll
            for (int u = 0; u < U; u++) any_slow |= slow[u];
#ifdef DTR_PROFILE
            {
                int32_t ns = 0;
#pragma unroll
                for (int u = 0; u < U; u++) ns += slow[u] ? 1 : 0;
                s.prof_slow += ns;     // per lane; reduced at the end
                for (int u = 0; u < U; u++) s.prof_global_nodes += ok[u] && (pd[u] & 0xFF) > K ? 1 : 0;
            }
#endif
            if (__ballot(any_slow)) {
                if (lds_nodes) {
                    LdsNodes NL;
                    NL.p = s.S.nodes.lds_l;
#pragma unroll
                    for (int u = 0; u < U; u++)
                        if (slow[u]) sum[u] = eq_cost_full(s, NL, ab[u], ab[u] + (pd[u] >> 8), ev[u], bad);
                } else {
                    AnyNodes NA;
                    NA.n = s.S.nodes;
#pragma unroll
                    for (int u = 0; u < U; u++)
                        if (slow[u]) sum[u] = eq_cost_full(s, NA, ab[u], ab[u] + (pd[u] >> 8), ev[u], bad);
                }
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                N[u] = (uint64_t)(c0[u] + sum[u]);
                DA[u] = s.use_m ? (uint64_t)size[u] : 1;
                DB[u] = s.use_s ? (uint64_t)(T - last[u]) : 1;
                s.nbr += ok[u] ? ev[u] : 0;
                s.adj += ok[u] ? (pd[u] >> 8) : 0;
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; u++) {
                if (s.cmode == CM_RAND) {
                    const uint64_t key = ((uint64_t)s.evict_no << 32) + (uint64_t)(uint32_t)id[u];
                    N[u] = mix64(s.seed + 0x9E3779B97F4A7C15ull * key);
                    DA[u] = DB[u] = 1;
                } else {
                    N[u] = s.cmode == CM_LOCAL ? (uint64_t)c0[u] : 1;
                    DA[u] = s.use_m ? (uint64_t)size[u] : 1;
                    DB[u] = s.use_s ? (uint64_t)(T - last[u]) : 1;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            take(best, ok[u], score_est(N[u], DA[u], DB[u]), N[u], DA[u], DB[u], id[u], (int32_t)slot[u]);
            if (approx(HC)) scored += __popcll(__ballot(ok[u]));
        }
    }
}

template <int HC>
__device__ __forceinline__ int32_t scan(Sim &s, int32_t &victim_slot, const Filter &F, int64_t &scored)
{
    bool bad = false;
    Best best;
    best.sc = best.lo = best.hi = 0.0f;
    best.N = 0;
    best.da = best.db = 1;
    best.id = 0x7fffffff;
    best.slot = -1;
    best.have = 0;
    if constexpr (cls(HC) == HC_WALK) walk_scan<HC>(s, F, best, scored);
    else scan_rounds<HC>(s, F, best, scored, bad);
    if (__ballot(bad)) { set_status(s, ST_CAPACITY); return -1; }
    // cross-lane minimum: the smallest estimate bounds the winner; only the
    // lanes within the filter margin of it (usually one) are compared exactly
    float mn = best.have ? best.sc : __builtin_inff();
    for (int off = WAVE / 2; off >= 1; off >>= 1) mn = fminf(mn, __shfl_xor(mn, off, WAVE));
    const float thr = mn * FILTER_HI;
    uint64_t m = __ballot(best.have && !(best.sc > thr));     // NaN estimates stay in
    if (!m) return -1;
    int32_t j = __ffsll((long long)m) - 1;
    m &= m - 1;
    uint64_t wN = readlane64(best.N, j), wda = readlane64(best.da, j), wdb = readlane64(best.db, j);
    int32_t wid = __builtin_amdgcn_readlane(best.id, j), wslot = __builtin_amdgcn_readlane(best.slot, j);
    while (m) {
        j = __ffsll((long long)m) - 1;
        m &= m - 1;
        const uint64_t cN = readlane64(best.N, j), cda = readlane64(best.da, j), cdb = readlane64(best.db, j);
        const int32_t cid = __builtin_amdgcn_readlane(best.id, j), cslot = __builtin_amdgcn_readlane(best.slot, j);
        if (better_exact(cN, cda, cdb, cid, wN, wda, wdb, wid)) {
            wN = cN;
            wda = cda;
            wdb = cdb;
            wid = cid;
            wslot = cslot;
        }
    }
    victim_slot = wslot;
    return wid;
}

// ----------------------------------------------------- operator calls --

template <int HC>
__device__ __forceinline__ bool allocate(Sim &s, int64_t sz)
{
    while (s.mem + sz > s.budget) {
        if (s.pool_live == 0) { set_status(s, ST_OOM); return false; }
        // keep the scanned range within half a round of the live pool
        if (s.pool_end > s.pool_live + WAVE * Round<HC>::value / 2) pool_compact<HC>(s);
#ifdef DTR_PROFILE
        const int64_t c0_ = (int64_t)__builtin_readcyclecounter();
        s.prof_scans++;
        if (cls(HC) != HC_WALK) s.prof_rounds += (s.pool_end + WAVE * Round<HC>::value - 1) / (WAVE * Round<HC>::value);
#endif
        int32_t slot = -1;
        int64_t scored = 0;
        Filter F;
        F.sample = false;
        F.min_size = F.tau = 0;
        if (approx(HC)) F = make_filter<HC>(s);
        int32_t v;
        for (;;) {
            v = scan<HC>(s, slot, F, scored);
            if (v >= 0 || !F.sample || s.status != ST_OK) break;
            F.sample = false;      // the sample missed every candidate that is not small: search those
        }
#ifdef DTR_PROFILE
        s.prof_scan_cycles += (int64_t)__builtin_readcyclecounter() - c0_;
#endif
        if (v < 0) { set_status(s, ST_CAPACITY); return false; }
        s.scores += approx(HC) ? scored : s.pool_live;
        PROF_T0(te);
        const bool evicted = evict<HC>(s, v, slot, false);
        PROF_ADD(PH_EVICT, te);
        if (!evicted) return false;
        s.evict_no++;
    }
    return true;
}

// Frame of the explicit rematerialization stack: while a frame is current,
// lane k holds input k's id and state word (operations with more inputs than
// lanes use the chunked path).
struct Frame {
    int32_t u;        // this lane's input (or -1)
    uint64_t w;       // its state word, lock included
};

// lock inputs ids[b..e) (one lane per input); tensors that were evictable
// leave the pool.  Fills f for single-chunk operations.
// `head`: when >= -1, lanes below NB_HEAD hold the first entries of ids[b..)
// already (an operation's inputs are the first neighbours of its output)
__device__ __forceinline__ void lock_inputs(Sim &s, const int32_t *ids, int32_t b, int32_t e, Frame &f,
                                            int32_t head = -2)
{
    for (int32_t k0 = b; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        bool killed = false;
        int32_t u = -1;
        uint64_t nw = 0;
        if (k < e) {
            u = head >= -1 && k0 == b && s.lane < NB_HEAD ? head : gld(ids + k);
            const uint64_t w = s.S.tst[u];
            const uint32_t l = ts_locks(w);
            // counts from LOCKS_SAT on are kept in lockx (the field stays saturated)
            nw = l < LOCKS_SAT ? ts_make(ts_sw(w), ts_pos(w), l + 1) : w;
            if (l + 1 == LOCKS_SAT) s.S.lockx[u] = (int32_t)LOCKS_SAT;
            else if (l == LOCKS_SAT) s.S.lockx[u] = s.S.lockx[u] + 1;
            if (ts_in_pool(w)) {
                s.S.pool((int32_t)ts_pos(w)).id = -1;
                killed = true;
            }
            s.S.tst[u] = nw;
        }
        if (k0 == b) {
            f.u = u;
            f.w = nw;
        }
        s.pool_live -= __popcll(__ballot(killed));
    }
}

// reload a frame's inputs after returning from nested rematerializations;
// lanes below NB_HEAD have their input id from the stack frame already (u8)
__device__ __forceinline__ void reload_frame(const Sim &s, int32_t b, int32_t e, Frame &f, int32_t u8)
{
    const int32_t k = b + s.lane;
    f.u = k < e ? (s.lane < NB_HEAD ? u8 : gld(s.t.in + k)) : -1;
    f.w = f.u >= 0 ? s.S.tst[f.u] : 0;
}

// unlock inputs [b, e); tensors left unlocked and resident rejoin the pool
// with last access `last`
template <int HC>
__device__ __forceinline__ void unlock_inputs(Sim &s, int32_t b, int32_t e, int64_t last, const Frame &f)
{
    for (int32_t k0 = b; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        int32_t u = -1;
        uint64_t w = 0;
        if (k < e) {
            if (k0 == b) {
                u = f.u;
                w = f.w;
            } else {
                u = gld(s.t.in + k);
                w = s.S.tst[u];
            }
        }
        const uint32_t l = ts_locks(w);
        const bool join = k < e && l == 1 && ts_sw(w) == S_RESIDENT;
        const int32_t slot = pool_append<HC>(s, join, u, last);
        if (k < e) {
            uint32_t nl = l - 1;
            if (l == LOCKS_SAT) {
                // a saturated count leaves lockx once it drops below LOCKS_SAT
                const int32_t c = s.S.lockx[u] - 1;
                if (c >= (int32_t)LOCKS_SAT) {
                    s.S.lockx[u] = c;
                    nl = LOCKS_SAT;
                }
            }
            s.S.tst[u] = ts_make(ts_sw(w), join ? (uint32_t)slot : ts_pos(w), nl);
        }
    }
}

// index (relative to b) of the first evicted input at or after `from`, or e - b
__device__ __forceinline__ int32_t next_evicted(const Sim &s, int32_t b, int32_t e, int32_t from, const Frame &f)
{
    const bool ev0 = s.lane >= from && b + s.lane < e && ts_sw(f.w) >= 0;
    const uint64_t m0 = __ballot(ev0);
    if (m0) return __ffsll((long long)m0) - 1;
    for (int32_t k0 = b + WAVE; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        bool ev = false;
        if (k < e && k - b >= from) ev = ts_sw(s.S.tst[gld(s.t.in + k)]) >= 0;
        const uint64_t m = __ballot(ev);
        if (m) return k0 - b + __ffsll((long long)m) - 1;
    }
    return e - b;
}

// run the parent operation of t (record rt); its start time is the last
// access of its inputs and output
template <int HC>
__device__ __forceinline__ bool execute(Sim &s, int32_t t, const TRec &rt, bool remat, uint32_t locks)
{
    const int64_t c = rt.c0;
    s.T += c;
    s.total += c;
    s.executed++;
    if (cls(HC) == HC_WALK && (s.executed & (PROGRESS_STEP - 1)) == 0 && s.lane == 0)
        atomicAdd(s.progress, (unsigned long long)PROGRESS_STEP);
    if (remat) { s.remats++; s.remat_cost += c; }
    else s.base += c;
    s.mem += rt.size;
    if (s.mem > s.peak) s.peak = s.mem;
    if (cls(HC) == HC_EQ && remat) {
        const int32_t head = gld(s.t.rec[t].nb + (s.lane & (NB_HEAD - 1)));
        // split approximation: the set loses c0(t); t leaves it (its node stays as a phantom)
        const int32_t old = uni(ts_sw(s.S.tst[t]));
        if (s.uf_n <= UF_LDS) {
            LdsNodes NL;
            NL.p = s.S.nodes.lds_l;
            const int32_t r = find_compress(s, NL, old);
            NL.set_cost(r, uni64(NL.cost(r)) - c);
        } else {
            AnyNodes NA;
            NA.n = s.S.nodes;
            const int32_t r = find_compress(s, NA, old);
            NA.set_cost(r, uni64(NA.cost(r)) - c);
        }
        bool lost = false;
        for (int32_t k0 = rt.adj_b; k0 < rt.adj_e; k0 += WAVE) {
            const int32_t k = k0 + s.lane;
            if (k < rt.adj_e) {
                const uint64_t wx = s.S.tst[k0 == rt.adj_b && s.lane < NB_HEAD ? head : gld(s.t.adj + k)];
                if (ts_in_pool(wx) && !list_remove(s, (int32_t)ts_pos(wx), old)) lost = true;
            }
        }
        if (__ballot(lost)) set_status(s, ST_CAPACITY);
    }
    s.S.tst[t] = ts_make(S_RESIDENT, 0, locks);
    if (s.T >= CLOCK_LIMIT) { set_status(s, ST_CLOCK); return false; }
    return s.status == ST_OK;
}

// Banish t (Appendix C.4) unless one of its children is evicted or an
// operation in progress holds it, in which case it stays pending: its memory
// is reclaimed if resident (constants included), it is gone for good, and its
// resident children are pinned (never evictable).  Counted with the eager
// evictions.
__device__ __forceinline__ void try_banish(Sim &s, int32_t t)
{
    const uint64_t w = (uint64_t)uni64((int64_t)s.S.tst[t]);
    const int32_t b = uni(cld(s.t.ch_off + t)), e = uni(cld(s.t.ch_off + t + 1));
    bool blocked = ts_locks(w) > 0;
    for (int32_t k0 = b; k0 < e && !blocked; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        const bool ev = k < e && ts_sw(s.S.tst[gld(s.t.ch + k)]) >= 0;
        blocked = __ballot(ev) != 0;
    }
    if (blocked) {
        if (s.lane == 0) s.S.pending[t] = 1;
        return;
    }
    if (s.lane == 0) s.S.pending[t] = 0;
    const int32_t sw = ts_sw(w);
    if (sw == S_RESIDENT || sw == S_PINNED || sw == S_CONST) s.mem -= rec_u(s, t).size;
    if (ts_in_pool(w)) {
        if (s.lane == 0) s.S.pool((int32_t)ts_pos(w)).id = -1;
        s.pool_live--;
    }
    s.S.tst[t] = ts_make(S_BANISHED, 0, 0);
    s.eager++;
    for (int32_t k0 = b; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        bool killed = false;
        if (k < e) {
            const int32_t c = gld(s.t.ch + k);
            const uint64_t wc = s.S.tst[c];
            if (ts_sw(wc) == S_RESIDENT) {
                killed = ts_in_pool(wc);
                if (killed) s.S.pool((int32_t)ts_pos(wc)).id = -1;
                s.S.tst[c] = ts_make(S_PINNED, ts_pos(wc), ts_locks(wc));
            }
        }
        s.pool_live -= __popcll(__ballot(killed));
    }
}

// after a rematerialization by the operation with inputs [b, e): the new
// tensor is a child of each input, so pending inputs retry banishing (in
// listed order)
__device__ __forceinline__ void retry_banish(Sim &s, int32_t b, int32_t e)
{
    for (int32_t k0 = b; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        int32_t p = -1;
        bool pend = false;
        if (k < e) {
            p = gld(s.t.in + k);
            pend = s.S.pending[p] != 0;
        }
        uint64_t m = __ballot(pend);
        while (m) {
            const int32_t j = __ffsll((long long)m) - 1;
            m &= m - 1;
            try_banish(s, __builtin_amdgcn_readlane(p, j));
        }
    }
}

constexpr int FQ = (int)(sizeof(StackFrame) / 16);    // 16-byte quads per stack frame

// push the current frame (tensor t, next input to check, its record); lane k
// below NB_HEAD saves its input id u
__device__ __forceinline__ void stack_push(const Sim &s, int32_t sp, int32_t t, int32_t next, const TRec &r, int32_t u)
{
    GAS i32x4 *F = s.S.stack + FQ * (size_t)sp;
    if (s.lane < NB_HEAD) ((GAS int32_t *)(F + 3))[s.lane] = u;
    i32x4 a, b, c;
    a.x = t;
    a.y = next;
    a.z = a.w = 0;
    b.x = (int32_t)(uint32_t)(uint64_t)r.size;
    b.y = (int32_t)(uint32_t)((uint64_t)r.size >> 32);
    b.z = r.c0;
    b.w = r.producer;
    c.x = r.in_b;
    c.y = r.in_e;
    c.z = r.adj_b;
    c.w = r.adj_e;
    F[0] = a;
    F[1] = b;
    F[2] = c;
}

__device__ __forceinline__ void stack_pop(const Sim &s, int32_t sp, int32_t &t, int32_t &next, TRec &r, int32_t &u8)
{
    const GAS i32x4 *F = s.S.stack + FQ * (size_t)sp;
    u8 = s.lane < NB_HEAD ? ((const GAS int32_t *)(F + 3))[s.lane] : -1;
    const i32x4 a = F[0], b = F[1], c = F[2];
    t = uni(a.x);
    next = uni(a.y);
    r.size = uni64((int64_t)(((uint64_t)(uint32_t)b.y << 32) | (uint32_t)b.x));
    r.c0 = uni(b.z);
    r.producer = uni(b.w);
    r.in_b = uni(c.x);
    r.in_e = uni(c.y);
    r.adj_b = uni(c.z);
    r.adj_e = uni(c.w);
}

// Run the operation producing `root` together with every rematerialization it
// needs (explicit stack instead of recursion).  root_remat: the root itself is
// a rematerialization held by the output condition.  Returns false once the
// simulation has stopped.
template <int HC>
__device__ __forceinline__ bool call(Sim &s, int32_t root, bool root_remat, uint32_t root_locks)
{
    int32_t sp = 0;
    int32_t tt = root, cur = -1;
    uint32_t tlocks = root_locks;     // locks held on tt by the frame below
    bool remat = root_remat;
    Frame f;
    f.u = -1;
    f.w = 0;
    TRec rt = rec_u(s, tt);           // record of the current frame's tensor
    // its first inputs, read alongside the record (their addresses need only tt)
    int32_t head = gld(s.t.rec[tt].nb + (s.lane & (NB_HEAD - 1)));
    for (;;) {
        PROF_T0(td);
        const int32_t b = rt.in_b, e = rt.in_e;
        if (cur < 0) {
            PROF_T0(tl);
            lock_inputs(s, s.t.in, b, e, f, head);
            PROF_ADD(PH_LOCK, tl);
            if (s.status != ST_OK) return false;
            cur = 0;
        }
        const int32_t j = uni(next_evicted(s, b, e, cur, f));
        PROF_ADD(PH_DESCEND, td);
        if (j < e - b) {
            if (sp + 1 >= s.S.n_max) { set_status(s, ST_CAPACITY); return false; }
            const int32_t child = j < WAVE ? __builtin_amdgcn_readlane(f.u, j) : uni(cld(s.t.in + b + j));
            const uint32_t clocks = j < WAVE ? ts_locks(readlane64(f.w, j))
                                             : (uint32_t)uni((int32_t)ts_locks(s.S.tst[child]));
            stack_push(s, sp, tt, j + 1, rt, f.u);
            sp++;
            tt = child;
            tlocks = clocks;
            cur = -1;
            remat = true;
            rt = rec_u(s, tt);
            head = gld(s.t.rec[tt].nb + (s.lane & (NB_HEAD - 1)));
            continue;
        }
        if (!allocate<HC>(s, rt.size)) return false;
        const int64_t start = s.T;
        PROF_T0(tx);
        const bool done = execute<HC>(s, tt, rt, remat, tlocks);
        PROF_ADD(PH_EXECUTE, tx);
        if (!done) return false;
        PROF_T0(tu);
        unlock_inputs<HC>(s, b, e, start, f);
        PROF_ADD(PH_UNLOCK, tu);
        if (cls(HC) != HC_EQ && remat && s.policy == POLICY_BANISH) retry_banish(s, b, e);
        if (!remat) {
            // a trace operation's output is unlocked: it joins the pool at once
            PROF_T0(to);
            const int32_t slot = uni(pool_append<HC>(s, s.lane == 0, tt, start, &rt));
            s.S.tst[tt] = ts_make(S_RESIDENT, (uint32_t)slot, 0);
            PROF_ADD(PH_OUTPUT, to);
        }
        if (s.status != ST_OK) return false;
        if (sp == 0) return true;
        PROF_T0(tr);
        sp--;
        int32_t u8;
        stack_pop(s, sp, tt, cur, rt, u8);
        remat = sp > 0 ? true : root_remat;
        reload_frame(s, rt.in_b, rt.in_e, f, u8);
        // locks on the resumed frame's output: none for a trace operation,
        // else whatever its consumers (or the output condition) hold
        tlocks = remat ? (uint32_t)uni((int32_t)ts_locks(s.S.tst[tt])) : 0u;
        PROF_ADD(PH_RESUME, tr);
    }
}

// what happens to the tensors released after op o (ascending id): eager
// eviction, nothing, or banishing
template <int HC>
__device__ __forceinline__ bool release(Sim &s, int32_t o)
{
    const int32_t b = uni(cld(s.t.rel_off + o)), e = uni(cld(s.t.rel_off + o + 1));
    if (s.policy == POLICY_IGNORE) return true;
    if (cls(HC) != HC_EQ && s.policy == POLICY_BANISH) {    // never a union-find heuristic
        for (int32_t k = b; k < e; k++) try_banish(s, uni(cld(s.t.rel + k)));
        return true;
    }
    for (int32_t k0 = b; k0 < e; k0 += WAVE) {
        const int32_t k = k0 + s.lane;
        int32_t r = -1, pos = 0;
        bool ev = false;
        if (k < e) {
            r = gld(s.t.rel + k);
            const uint64_t w = s.S.tst[r];
            ev = ts_in_pool(w);
            pos = (int32_t)ts_pos(w);
        }
        uint64_t m = __ballot(ev);
        while (m) {
            const int32_t j = __ffsll((long long)m) - 1;
            m &= m - 1;
            if (!evict<HC>(s, __builtin_amdgcn_readlane(r, j), __builtin_amdgcn_readlane(pos, j), true)) return false;
        }
    }
    return true;
}

template <int HC>
__device__ __forceinline__ void run_sim(const KernelArgs &a, int32_t sim, const Slot &S, int32_t lane, LAS WalkCtl *ctl,
                                       int32_t nw)
{
    Sim s;
    const SpecDev sp = a.specs[sim];
    s.t = a.traces[sp.trace];
    s.S = S;
    s.trace_idx = sp.trace;
    s.progress = a.progress;
    s.nw = nw;
    s.ctl = ctl;
    s.h = sp.heuristic;
    s.policy = sp.policy;
    s.search = sp.search;
    if (s.h >= H_FAMILY) {             // h'(s, m, c) = 16 + 4c + 2s + m
        s.cmode = (s.h - H_FAMILY) >> 2;
        s.use_s = (s.h >> 1) & 1;
        s.use_m = s.h & 1;
    } else {
        // the named heuristics as members of the family (Section 4.1, Appendix
        // A.3), packed 3 bits of cost measure and one bit of each flag per id
        constexpr uint32_t CM = CM_ESTAR | CM_EQCLASS << 3 | CM_LOCAL << 6 | CM_NONE << 9 | CM_NONE << 12 |
                                CM_RAND << 15 | CM_ESTAR << 18 | CM_ANCESTORS << 21;
        constexpr uint32_t US = 0x0F;    // h_DTR, h_eq, h_local, h_LRU use staleness
        constexpr uint32_t UM = 0xD7;    // all but h_LRU and h_rand use size
        const int32_t k = s.h & 7;
        s.cmode = (int32_t)((CM >> (3 * k)) & 7);
        s.use_s = (int32_t)((US >> k) & 1);
        s.use_m = (int32_t)((UM >> k) & 1);
    }
    s.lane = lane;
    s.budget = sp.budget;
    s.seed = sp.seed;
    s.T = 0;
    s.pool_end = s.pool_live = 0;
    s.uf_n = 1;                          // node 0: the null node (h_DTR^eq)
    s.uf_limit = UF_LDS;
    s.status = ST_OK;
    s.cur_op = 0;
    s.evict_no = 0;
    s.total = s.base = s.remat_cost = s.executed = s.remats = s.evictions = s.eager = s.scores = 0;
    s.nbr = s.adj = 0;
#ifdef DTR_PROFILE
    const int64_t t_start = (int64_t)__builtin_readcyclecounter();
    s.prof_scan_cycles = s.prof_scans = s.prof_rounds = 0;
    s.prof_slow = s.prof_global_nodes = s.prof_uf_compact = s.prof_pool_compact = 0;
    for (int k = 0; k < PROF_PHASES; k++) s.prof_ph[k] = 0;
#endif

    const int32_t n = s.t.n;
    for (int32_t x = lane; x < n; x += WAVE)
        s.S.tst[x] = ts_make((gld(s.t.flags + x) & FLAG_CONST) ? S_CONST : S_UNCOMPUTED, 0, 0);
    if (cls(HC) != HC_EQ && s.policy == POLICY_BANISH)
        for (int32_t x = lane; x < n; x += WAVE) s.S.pending[x] = 0;
    if (cls(HC) == HC_EQ && lane == 0) {
        UfNode z;
        z.cost = 0;
        z.parent = 0;
        z.size = 1;
        s.S.nodes[0] = z;
    }
    slot_sync<HC>();
    s.mem = s.t.const_mem;
    s.peak = s.mem;

    bool ok = true;
    if (s.mem > s.budget) { set_status(s, ST_OOM); ok = false; }
    for (int32_t o = 0; ok && o < s.t.F; o++) {
        s.cur_op = o;
        if (!call<HC>(s, uni(cld(s.t.out + o)), false, 0)) ok = false;
        PROF_T0(tr);
        if (ok && (!release<HC>(s, o) || s.status != ST_OK)) ok = false;
        PROF_ADD(PH_RELEASE, tr);
    }
    if (ok) {
        // output condition: lock each required output, rematerialize it if evicted
        s.cur_op = s.t.F;
        for (int32_t k = 0; ok && k < s.t.n_req; k++) {
            Frame f;
            lock_inputs(s, s.t.req, k, k + 1, f);
            const int32_t r = uni(cld(s.t.req + k));
            const uint64_t w = readlane64(f.w, 0);
            if (s.status != ST_OK) ok = false;
            else if (ts_sw(w) >= 0 && !call<HC>(s, r, true, (uint32_t)uni((int32_t)ts_locks(w)))) ok = false;
        }
    }

    int64_t nbr = s.nbr, adj = s.adj;
    for (int off = WAVE / 2; off >= 1; off >>= 1) {
        nbr += __shfl_xor(nbr, off, WAVE);
        adj += __shfl_xor(adj, off, WAVE);
    }
#ifdef DTR_PROFILE
    for (int off = WAVE / 2; off >= 1; off >>= 1) {
        s.prof_slow += __shfl_xor(s.prof_slow, off, WAVE);
        s.prof_global_nodes += __shfl_xor(s.prof_global_nodes, off, WAVE);
    }
    if (lane == 0 && a.prof) {
        int64_t *pr = a.prof + (size_t)sim * PROF_FIELDS;
        pr[0] = (int64_t)__builtin_readcyclecounter() - t_start;
        pr[1] = s.prof_scan_cycles;
        pr[2] = s.prof_scans;
        pr[3] = s.prof_rounds;
        pr[4] = s.prof_slow;
        pr[5] = s.prof_global_nodes;
        pr[6] = s.prof_uf_compact;
        pr[7] = s.prof_pool_compact;
        for (int k = 0; k < PROF_PHASES; k++) pr[8 + k] = s.prof_ph[k];
    }
#endif
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
    if (s.nw > 1) {
        // release the helper wavefronts from this simulation
        if (lane == 0) ctl->cmd = CMD_DONE;
        __syncthreads();
    } else {
        slot_sync<HC>();
    }
}

// The exact h_DTR^eq kernel: every wavefront takes simulations from the work
// counter on its own, in its own slot and LDS arrays, with no workgroup
// barrier (four to a workgroup: LDS is allocated per workgroup, so one
// allocation serves four simulations).
template <int HC>
__device__ __forceinline__ void eq_waves(const KernelArgs &a, UfNode *lds_nodes, PoolSlotL *lds_pool, int32_t lane,
                                         int32_t wave)
{
    const int32_t slot = (int32_t)blockIdx.x * lds_waves(HC) + wave;
    if (slot >= a.n_slots) return;
    Slot S = slot_at(a, slot);
    S.nodes.lds = lds_nodes + wave * UF_LDS;
    S.nodes.lds_l = (LAS UfNode *)lds_nodes + wave * UF_LDS;
    S.lpool = lds_pool + wave * POOL_LDS;
    S.lpool_l = (LAS PoolSlotL *)lds_pool + wave * POOL_LDS;
    for (;;) {
        uint32_t k = 0;
        if (lane == 0) k = atomicAdd(a.queue, 1u);
        k = (uint32_t)uni((int32_t)k);
        if (k >= (uint32_t)a.n_sims) break;
        run_sim<HC>(a, a.order[k], S, lane, nullptr, 1);
    }
}

// One simulation per workgroup at a time, taken from the work counter (the
// exact h_DTR^eq kernel: one per wavefront, as above).  The workgroups of the
// walk heuristics may hold helper wavefronts (a.L.walk_waves in all) that
// join the simulating wavefront's walk scans; every wavefront learns the next
// simulation from the control block after a workgroup barrier, so all of them
// leave the loop together.
template <int HC>
__global__ void __launch_bounds__(cls(HC) == HC_WALK ? MAX_WALK_WAVES * WAVE : lds_waves(HC) * WAVE)
    __attribute__((amdgpu_waves_per_eu(2))) replay_kernel(KernelArgs a)
{
    constexpr int LW = lds_waves(HC);
    // union-find nodes (h_DTR^eq: one array per wavefront), or the walk
    // control block (walk heuristics)
    __shared__ UfNode lds_nodes[cls(HC) == HC_EQ ? UF_LDS * LW : CTL_NODES];
    __shared__ PoolSlotL lds_pool[POOL_LDS * LW];
    const int32_t lane = (int32_t)threadIdx.x & (WAVE - 1);
    const int32_t wave = uni((int32_t)threadIdx.x / WAVE);
    if constexpr (LW > 1) {
        eq_waves<HC>(a, lds_nodes, lds_pool, lane, wave);
        return;
    }
    const int32_t nw = cls(HC) == HC_WALK ? (int32_t)a.L.walk_waves : 1;
    Slot S = slot_at(a, blockIdx.x);
    S.nodes.lds = lds_nodes;
    S.nodes.lds_l = (LAS UfNode *)lds_nodes;
    S.lpool = lds_pool;
    S.lpool_l = (LAS PoolSlotL *)lds_pool;
    LAS WalkCtl *ctl = (LAS WalkCtl *)lds_nodes;
    if (cls(HC) == HC_WALK) {
        // visited bitmaps start clear (every walk clears what it set)
        // (the flags 16 bytes at a time: vis_bytes is a multiple of 16)
        GAS u32x4 *V = (GAS u32x4 *)(S.visb + (size_t)(wave * WAVE) * (size_t)S.vis_bytes);
        for (size_t i = lane; i < (size_t)WAVE * (size_t)S.vis_bytes / 16; i += WAVE) V[i] = u32x4{0u, 0u, 0u, 0u};
        GAS uint32_t *B = S.bigvis + (size_t)wave * (size_t)S.vis_words;
        for (int32_t i = lane; i < S.vis_words; i += WAVE) B[i] = 0u;
        wave_sync();
    }
    for (;;) {
        uint32_t k = 0;
        if (wave == 0 && lane == 0) k = atomicAdd(a.queue, 1u);
        if (nw > 1) {
            if (wave == 0 && lane == 0) ctl->sim = (int32_t)k;
            __syncthreads();
            k = (uint32_t)uni(ctl->sim);
        } else {
            k = (uint32_t)uni((int32_t)k);
        }
        if (k >= (uint32_t)a.n_sims) break;
        if constexpr (cls(HC) == HC_WALK) {
            if (wave == 0) run_sim<HC>(a, a.order[k], S, lane, ctl, nw);
            else help_walks<HC>(a, S, lane, wave, ctl);
        } else {
            run_sim<HC>(a, a.order[k], S, lane, ctl, 1);
        }
    }
}

__global__ void reset_kernel(uint32_t *queue, int32_t n)
{
    if ((int32_t)threadIdx.x < n) queue[threadIdx.x] = 0;
}

// Working memory of dtr_sim_run_static: the work counters (first 256 bytes),
// then the simulation slots.  One copy per device, held until the process
// ends; every static run on a device shares it.
constexpr size_t STATIC_SCRATCH_BYTES = DTR_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[STATIC_SCRATCH_BYTES];

}  // namespace dtr

// Device address and size of this device's static working memory.  The
// address is looked up once per device (with that device current) and kept:
// in host code the array's name is not a device address.
extern "C" hipError_t dtr_static_scratch(void **ptr, size_t *bytes)
{
    constexpr int MAX_DEVICES = 64;
    static std::mutex mu;
    static void *addr[MAX_DEVICES] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(dtr::scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    *bytes = dtr::STATIC_SCRATCH_BYTES;
    return hipSuccess;
}

// Launch entries used by the host library (same shared object): the work
// counters of the groups are cleared by a kernel, then each group g (heuristic
// class: union-find; neighbourhood walk; none; + 3 with the search
// approximations) runs its own kernel specialisation, each on the stream the
// host gives it (the groups use disjoint slots, so they may run at once).
extern "C" hipError_t dtr_launch_reset(uint32_t *queue, hipStream_t stream)
{
    using namespace dtr;
    hipLaunchKernelGGL(reset_kernel, dim3(1), dim3(WAVE), 0, stream, queue, COUNTER_WORDS);
    return hipGetLastError();
}

extern "C" hipError_t dtr_launch_group(const dtr::KernelArgs *a, int32_t group, hipStream_t stream)
{
    using namespace dtr;
    if (a->n_sims <= 0) return hipSuccess;
    const dim3 grid(a->n_slots), blk(WAVE), wblk(WAVE * (uint32_t)a->L.walk_waves);
    // the exact h_DTR^eq kernel: EQ_WAVES slots per workgroup
    const dim3 egrid((a->n_slots + EQ_WAVES - 1) / EQ_WAVES), eblk(WAVE * EQ_WAVES);
    switch (group) {
    case 0: hipLaunchKernelGGL(replay_kernel<HC_EQ>, egrid, eblk, 0, stream, *a); break;
    case 1: hipLaunchKernelGGL(replay_kernel<HC_WALK>, grid, wblk, 0, stream, *a); break;
    case 2: hipLaunchKernelGGL(replay_kernel<HC_SIMPLE>, grid, blk, 0, stream, *a); break;
    case 3: hipLaunchKernelGGL(replay_kernel<HC_EQ | HC_APPROX>, grid, blk, 0, stream, *a); break;
    case 4: hipLaunchKernelGGL(replay_kernel<HC_WALK | HC_APPROX>, grid, wblk, 0, stream, *a); break;
    case 5: hipLaunchKernelGGL(replay_kernel<HC_SIMPLE | HC_APPROX>, grid, blk, 0, stream, *a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}
