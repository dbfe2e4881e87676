// layout.h -- device-side tables of the batched DTR replay, shared by the host
// library (dtr_sim.cpp, which derives and uploads them) and the kernels
// (replay.hip).  Everything lives in the caller's workspace.
#pragma once
#include <stdint.h>

namespace dtr {

// state word per tensor (sw[]): evicted tensors hold a non-negative value
// (their union-find node under h_DTR^eq, 0 otherwise)
constexpr int32_t SW_UNCOMPUTED = -2;
constexpr int32_t SW_RESIDENT = -1;

constexpr int64_t CLOCK_LIMIT = int64_t(1) << 40;
constexpr int WAVE = 64;

// Static per-trace tables (read-only during a run).  Derived on the host:
//   producer/c0      parent operation of each tensor and its cost (Appendix C.2)
//   adj              parents then children of each tensor: the undirected
//                    neighbourhood used by union-find components and the first
//                    ring of e*
//   ch               children: tensors whose parent operation reads the tensor
//   rel              tensors released after each op (last reader), ascending id
//   req / consts     required outputs and constants, ascending id
// Per-tensor static record, one scalar load (32 bytes): size, c0, parent
// operation, its input range in `in`, and the tensor's neighbour range in `adj`.
constexpr int NB_HEAD = 8;

struct TRec {
    int64_t size;
    int32_t c0;              // cost of the parent operation (<= 2^28), 0 for constants
    int32_t producer;        // -1 for constants
    int32_t in_b, in_e;      // inputs of the parent operation
    int32_t adj_b, adj_e;    // parents then children
};
static_assert(sizeof(TRec) == 32, "tensor record layout");
// The record array's element: the record, then the tensor's first NB_HEAD
// neighbours in `adj` order (its parent operation's inputs first), padded
// with tensor 0.  The record alone is one 32-byte scalar load; the neighbour
// ids are addressed by the tensor id alone.
struct TRecX {
    TRec r;
    int32_t nb[NB_HEAD];
};
static_assert(sizeof(TRecX) == 64, "tensor record element layout");

struct TraceDev {
    int32_t n;               // tensors
    int32_t F;               // ops
    int32_t n_req, n_const;
    int64_t const_mem;       // memory held by constants
    const int64_t *size;     // [n]
    const int64_t *c0;       // [n]
    const uint8_t *flags;    // [n]
    const int32_t *producer; // [n]  -1 for constants
    const int32_t *out;      // [F]
    const int64_t *cost;     // [F]
    const int32_t *in_off;   // [F+1]
    const int32_t *in;       // [E]
    const int32_t *ch_off;   // [n+1]
    const int32_t *ch;       // [E]
    const int32_t *adj_off;  // [n+1]
    const int32_t *adj;      // [2E]
    const int32_t *rel_off;  // [F+1]
    const int32_t *rel;      // [<= n]
    const int32_t *req;      // [n_req]
    const int32_t *consts;   // [n_const]
    const TRecX *rec;        // [n]
};

struct SpecDev {
    int32_t trace, heuristic;
    int64_t budget;
    uint64_t seed;
    int32_t policy, search;
};
static_assert(sizeof(SpecDev) == 32, "spec layout");

struct ResultDev {
    int64_t total_cost, base_cost, remat_cost, peak_memory, final_memory;
    int64_t n_executed_ops, n_remats, n_evictions, n_eager_evictions, n_scores;
    int64_t n_nbr_visits, n_adj_visits;
    int32_t status, failed_op;
};
static_assert(sizeof(ResultDev) == 104, "result layout");

// Per-slot working memory: one slot per resident simulation, sized for the
// largest trace of the batch (n_max tensors).  Offsets in bytes from the slot
// base, each 256-byte aligned.
//   tst       per-tensor state word: state/union-find node (32 bits), pool
//             position (24 bits), lock count (8 bits; 255 = the count is in lockx)
//   lockx     per-tensor lock count of tensors held 255 times or more (a
//             weight read by every operation of a deep rematerialization
//             stack); read and written only while the 8-bit field is saturated
//   pool      evictable tensors, pcap 64-byte slots (dead slots are
//             tombstoned and squeezed out): id, packed (degree << 8 | n), last
//             access, size, c0, start of the neighbour range, and for
//             h_DTR^eq the union-find nodes of up to NB_CACHE evicted
//             neighbours (n = NB_CACHE + 1 marks an overflowed cache); for
//             the walk heuristics n is the parent count (255: at least 255)
//             and the cache holds the first NB_HEAD neighbours
//   nodes     union-find nodes {running cost, parent, size}
//   stack     rematerialization frames (tensor, next input, the tensor's record,
//             its first input ids)
//   vis/wq    lane-private visited flags (one byte per tensor) and member
//             queues (wq_cap entries) of the e* and e_R walks (h_DTR, h_{e*},
//             h_MSPS), for every lane of the workgroup
//   bigvis/bigq  each wavefront's visited bitmap and queue (n_max + 1
//             entries) for walks that outgrow a lane's queue, which a whole
//             wavefront then takes; ovf lists those candidates' pool slots
//   pending   one byte per tensor: released, banishing deferred (banishing policy)
constexpr int NB_CACHE = 8;
// union-find node ids below UF_LDS live in LDS (16 bytes each per wavefront),
// the rest in the slot's global node array
constexpr int UF_LDS = 512;
// pool slots below POOL_LDS live in LDS (64 bytes each, padded to 80, per
// wavefront), the rest in the slot's global pool array (which keeps the same
// indices); with 18 KB of LDS per h_DTR^eq wavefront a compute unit holds as
// many of them as its registers allow (two per SIMD)
constexpr int POOL_LDS = 128;
// wavefronts per workgroup of the exact h_DTR^eq kernel, each running its own
// simulations with its own LDS arrays
constexpr int EQ_WAVES = 4;

struct SlotLayout {
    int64_t bytes;           // stride between slots
    int64_t tst, lockx;
    int64_t pool;
    int64_t nodes, uf_remap;
    int64_t stack;
    int64_t vis, wq, bigvis, bigq, ovf;
    int64_t pending;
    int64_t pcap, ucap, n_max;
    int64_t vis_words;       // 32-bit words of one wavefront's visited bitmap (a multiple of 4)
    int64_t vis_bytes;       // bytes of one lane's visited flags (a multiple of 16)
    int64_t wq_cap;          // entries of one lane's member queue
    int64_t walk_waves;      // wavefronts per workgroup of the walk heuristics
};
// workgroups of the walk heuristics hold up to this many wavefronts: the
// first runs the simulation, the others join its eviction scans
constexpr int MAX_WALK_WAVES = 8;
// a lane's member queue holds at most this many entries (walks that need
// more are taken by a whole wavefront, a level at a time)
constexpr int WALK_QUEUE_CAP = 256;

struct __attribute__((aligned(16))) PoolSlot {
    int32_t id;              // tensor; -1 marks a dead slot
    int32_t deg;             // degree << 8 | cached neighbour count (walks: parent count)
    int64_t last;            // last access
    int64_t size;
    int32_t c0;              // <= 2^28
    int32_t adj_b;           // start of the tensor's neighbour range
    int32_t nb[NB_CACHE];    // cached union-find nodes of evicted neighbours (walks: first neighbours)
};
static_assert(sizeof(PoolSlot) == 64, "pool slot layout");

struct __attribute__((aligned(16))) StackFrame {
    int32_t t, next, pad0, pad1;
    TRec rec;
    int32_t in8[NB_HEAD];    // the frame's first NB_HEAD input ids (-1 past the last)
};
static_assert(sizeof(StackFrame) == 80, "stack frame layout");

struct __attribute__((aligned(16))) UfNode {
    int64_t cost;
    int32_t parent;
    int32_t size;
};

// simulation groups, one kernel specialisation each: heuristic class
// (union-find neighbourhood, neighbourhood walk, none), plus 3 with the
// search approximations on
constexpr int N_GROUPS = 6;
// work-counter block at the head of the working memory: one 32-bit counter
// per group, then (at byte PROGRESS_OFFSET) the 64-bit progress counter
constexpr int PROGRESS_OFFSET = 32;
constexpr int COUNTER_WORDS = PROGRESS_OFFSET / 4 + 2;
constexpr int PROGRESS_STEP = 4096;

struct KernelArgs {
    const TraceDev *traces;
    const SpecDev *specs;
    const int32_t *order;    // sims, longest first
    ResultDev *results;
    uint32_t *queue;         // work counter, zeroed before each run
    unsigned long long *progress;   // walk heuristics' executed operations, in steps of PROGRESS_STEP
    uint8_t *slots;
    SlotLayout L;
    int32_t n_sims;
    int32_t n_slots;
    int64_t *prof;           // DTR_PROFILE builds: PROF_FIELDS counters per sim
};

// In-kernel phase timers (DTR_PROFILE builds only): cycles spent per sim in
// the whole replay and in the eviction scans, and the number of scans.
constexpr int PROF_PHASES = 8;   // evict, execute, unlock, lock, release, resume, output, descend
constexpr int PROF_FIELDS = 8 + PROF_PHASES;   // total cycles, scan cycles, scans, scan rounds,
                                               // recounts, overflowed caches, node and pool
                                               // compactions, then cycles per phase

}  // namespace dtr
