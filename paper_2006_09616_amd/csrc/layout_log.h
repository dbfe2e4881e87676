// layout_log.h -- device-side tables of the operator-log replay, shared by the
// host lowering (dtr_log.cpp) and its kernel (replay_log.hip).  Everything
// lives in the caller's workspace.
#pragma once
#include <stdint.h>

#include "layout.h"

namespace dtr {

// A lowered operator log (read-only during a run).  Storages are the unit of
// eviction; tensors are a storage's root or views of it; operators may have
// several outputs.  CSR offsets are int32 (validated sizes).
struct LogProgDev {
    int32_t S, T, F, n_req;
    // storages
    const int64_t *s_size;        // [S]
    const int64_t *s_c0;          // [S] summed cost of the operators computing its tensors (end of log)
    const uint8_t *s_const;       // [S] constant (pinned from creation)
    const int32_t *par_off, *par; // storage graph: parents (distinct input storages of those operators)
    const int32_t *ch_off, *ch;   //   and children; each list in the order its edges are created
    const int32_t *dt_off, *dt;   // tensors computed from the storage outside it (banishing)
    // tensors
    const int32_t *t_storage;     // [T]
    const int32_t *t_op;          // [T]
    const uint8_t *t_alias;       // [T] a view of another tensor's storage
    // operators, in log order
    const int64_t *op_cost;       // [F]
    const int64_t *op_need;       // [F] summed size of its non-view outputs
    const int32_t *in_off, *in;   // input tensors, listed order
    const int32_t *ls_off, *ls;   // distinct input storages (locking)
    const int32_t *out_off, *out; // output tensors
    const int32_t *rel_off, *rel; // storages released after each operator, in log order
    const int32_t *req;           // [n_req] tensors still referenced at the end, ascending
    const int32_t *born_off, *born; // per operator: (parent, storage) edges its first run creates
};

// Per-slot working memory of the log replay, sized for the largest log of
// the batch.  Byte offsets from the slot base, 256-byte aligned.
//   state/pinned/pending   u8  [S_max]  storage state, never-evictable flag,
//                                       banishing deferred
//   locks, node            i32 [S_max]  holds by operators in progress; the
//                                       union-find node of an evicted storage
//   sgen, last             i64 [S_max]  residency generation; last access
//   gen                    i64 [T_max]  generation at which each tensor's
//                                       operator last ran
//   c0d, pcnt, ccnt        i64/i32/i32 [S_max]  costs and edge counts of the
//                                       storage graph created so far
//   uf_*                   [ucap]       union-find nodes (parent, set size,
//                                       running cost), the compaction map and
//                                       a cost staging array
//   mark                   u32 [ucap * WAVE]  lane-private epoch stamps of
//                                       union-find roots (h_DTR^eq)
//   wmark                  u32 [wm_words * WAVE] lane-private visited bitsets
//                                       of the walks, when not in LDS
//   queue                  i32 [(S_max + 2) * WAVE] lane-private walk queues
//   stack                  LogFrame [F_max + 2] operator calls in progress
struct LogSlotLayout {
    int64_t bytes;
    int64_t state, pinned, pending;
    int64_t locks, node;
    int64_t sgen, last;
    int64_t gen;
    int64_t uf_parent, uf_size, uf_remap, uf_cost, uf_tmp;
    int64_t c0d, pcnt, ccnt;          // the graph created so far (device-memory variant)
    int64_t mark, wmark, queue;
    int64_t stack;
    int64_t S_max, T_max, F_max, ucap, mcap;
};

// one operator call in progress: the operator, the next input to check, and
// whether it is a rematerialization
struct LogFrame {
    int32_t op, next, remat, pad;
};
static_assert(sizeof(LogFrame) == 16, "frame layout");

struct LogKernelArgs {
    const LogProgDev *progs;
    const SpecDev *specs;
    const int32_t *order;
    ResultDev *results;
    uint32_t *queue;
    uint8_t *slots;
    LogSlotLayout L;
    int32_t n_sims, n_slots;
    // walk state in LDS when lds_bytes > 0: byte offsets of the storage
    // states, the 64 visited bitsets and the storage graph (16-bit ids)
    int32_t lds_bytes, lds_state, lds_wm, lds_po, lds_co, lds_pa, lds_ca;
    // and for the walk scan: storage costs c0, the candidate list, 64
    // pending-storage stacks of LOG_LDS_STACK entries, the candidate counter
    int32_t lds_c0, lds_cand, lds_stk, lds_ctr;
    int32_t lds_sz, lds_last;  // storage sizes and last-access times
    int32_t lds_rsum, lds_rcnt;  // per listed candidate: walked cost, count
    int32_t lds_pcnt, lds_ccnt;  // edges created so far per storage
    int32_t wm_words;         // 32-bit words per visited bitset (a multiple of 4)
    // LDS variant: waves per workgroup (1 .. MAX_LOG_WAVES; the first replays,
    // the others help with walk scans) and the offset of the control words
    int32_t waves, lds_ctl;
};

constexpr int LOG_LDS_STACK = 32;
constexpr int MAX_LOG_WAVES = 4;

}  // namespace dtr
