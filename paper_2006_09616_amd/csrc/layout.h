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
};

struct SpecDev {
    int32_t trace, heuristic;
    int64_t budget;
    uint64_t seed;
};

struct ResultDev {
    int64_t total_cost, base_cost, remat_cost, peak_memory, final_memory;
    int64_t n_executed_ops, n_remats, n_evictions, n_eager_evictions, n_scores;
    int64_t n_nbr_visits, n_adj_visits;
    int32_t status, failed_op;
};
static_assert(sizeof(ResultDev) == 104, "result layout");

// Per-slot working memory: one slot per resident simulation.  Column arrays
// sized for the largest trace of the batch (n_max tensors).  Offsets in bytes
// from the slot base, each 256-byte aligned.
struct SlotLayout {
    int64_t bytes;           // stride between slots
    int64_t sw, locks, last, pos;            // per tensor
    int64_t pool_id, pool_last, pool_size, pool_c0;   // pool columns
    int64_t stack;           // remat frames: (tensor, cursor) int32 pairs
    int64_t uf_parent, uf_cost, uf_size, uf_remap;    // union-find (h_DTR^eq)
    int64_t uf_cap;          // nodes
    int64_t stamp, queue;    // per-lane neighbourhood walk (h_DTR, h_ESTAR)
    int64_t n_max;
};

struct KernelArgs {
    const TraceDev *traces;
    const SpecDev *specs;
    const int32_t *order;    // sims, longest first
    ResultDev *results;
    uint32_t *queue;         // work counter, zeroed before each run
    uint8_t *slots;
    SlotLayout L;
    int32_t n_sims;
    int32_t n_slots;
};

}  // namespace dtr
