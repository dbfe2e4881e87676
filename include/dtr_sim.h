/*
 * dtr_sim.h -- C ABI of the batched Dynamic Tensor Rematerialization
 * eviction-loop simulator for AMD Instinct MI355X (gfx950).
 *
 * The library replays operator traces under DTR's greedy online policy
 * (Kirisame et al., "Dynamic Tensor Rematerialization", ICLR 2021):
 *   - operator call (Section 2; Appendix C.4 "(Re)materialization"): lock the
 *     inputs, rematerialize evicted inputs recursively by replaying their
 *     parent operation, allocate the output, evicting while memory is
 *     insufficient, advance the clock by the operator cost, unlock;
 *   - eviction (Appendix C.4): the evictable pool is every resident tensor
 *     with no locks (Appendix C.1); every pool member is scored and the
 *     lowest score is evicted;
 *   - eager eviction when the program drops its last reference (Section 2
 *     "Deallocation", Appendix C.5);
 *   - output condition (Appendix C.6): required outputs are rematerialized
 *     and locked at the end.
 * Each simulation is one (trace, heuristic, budget, seed).  Thousands run as
 * independent work items on one GPU; all quantities are integers and every
 * result is exact (bit-identical to a plain sequential implementation).
 *
 * Conventions used by every entry point:
 *   - host pointers are read only during the call unless stated otherwise;
 *   - the device workspace is caller-owned device memory (for example a
 *     torch uint8 tensor); it must stay allocated while the handle lives;
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream);
 *   - functions return DTR_OK (0) or a negative DTR_E* code; the message of
 *     the last error on the calling thread is in dtr_sim_last_error();
 *   - a handle is not thread-safe; distinct handles are independent.
 */
#ifndef DTR_SIM_H
#define DTR_SIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes (return values) ---------------------------------------- */
#define DTR_OK      0
#define DTR_EINVAL  (-1)   /* null pointer, bad count, workspace too small      */
#define DTR_ETRACE  (-2)   /* trace or simulation spec fails validation         */
#define DTR_EHIP    (-3)   /* a HIP runtime call failed                         */
#define DTR_ESTATE  (-4)   /* call out of order (results before run)            */

/* ---- tensor flags ---------------------------------------------------------- */
#define DTR_FLAG_CONSTANT 1u  /* no producer; resident from time 0; never evicted
                                 (Section 2: constants cannot be evicted)         */
#define DTR_FLAG_REQUIRED 2u  /* never released; must be resident at the end
                                 (Appendix C.6 output condition)                  */

/* ---- heuristics (score = N/D, lowest evicted; Section 4.1, Appendix C.3) --- */
#define DTR_H_DTR   0  /* (c0 + sum c0 over e*) / (m s), exact evicted neighbourhood   */
#define DTR_H_EQ    1  /* (c0 + union-find neighbourhood cost) / (m s), split approx.  */
#define DTR_H_LOCAL 2  /* c0 / (m s)                                                  */
#define DTR_H_LRU   3  /* 1 / s                                                       */
#define DTR_H_SIZE  4  /* 1 / m                                                       */
#define DTR_H_RAND  5  /* fresh SplitMix64 draw per (seed, eviction number, id)       */
#define DTR_H_ESTAR 6  /* (c0 + sum c0 over e*) / m, the h_{e*} of Appendix A.3       */
#define DTR_H_MSPS  7  /* (c0 + sum c0 over e_R) / m, e_R = the evicted tensors that
                          rematerializing the candidate would recompute (Section 4.1) */
/* The ablation family of Appendix D: h'(s, m, c) = c / (m s), where staleness
 * s and size m are each used (1) or ablated (0: the measure is 1), and c is
 * one of the cost measures below.  DTR_H_FAMILY(DTR_C_ESTAR, 1, 1) is h_DTR,
 * (DTR_C_EQCLASS, 1, 1) h_DTR^eq, (DTR_C_LOCAL, 1, 1) h_local, (DTR_C_NONE, 1,
 * 0) h_LRU, (DTR_C_NONE, 0, 1) h_size and (DTR_C_ESTAR, 0, 1) h_{e*}. */
#define DTR_C_ESTAR   0  /* c0 + sum c0 over e*                    */
#define DTR_C_EQCLASS 1  /* c0 + union-find neighbourhood cost      */
#define DTR_C_LOCAL   2  /* c0                                      */
#define DTR_C_NONE    3  /* 1                                       */
#define DTR_H_FAMILY(c, s, m) (16 + 4 * (c) + 2 * (s) + (m))

#define DTR_BUDGET_UNLIMITED INT64_MAX

/* ---- per-simulation status (a result, not an error) ------------------------ */
#define DTR_STATUS_OK             0
#define DTR_STATUS_OOM            1  /* nothing evictable while memory is short    */
#define DTR_STATUS_CLOCK_OVERFLOW 2  /* clock reached 2^40 cost units              */
#define DTR_STATUS_CAPACITY       3  /* internal capacity exceeded (never expected) */

/*
 * An operator trace.  Tensors are 0..n_tensors-1, operators 0..n_ops-1 in
 * execution order; every operator produces exactly one tensor (Section 2
 * assumptions).  Layout: plain host arrays.
 *   tensor_size[n_tensors]     bytes (or units), 1 <= size < 2^36
 *   tensor_flags[n_tensors]    DTR_FLAG_* bits
 *   op_output[n_ops]           tensor produced by each op; every non-constant
 *                              tensor is produced exactly once, constants never
 *   op_cost[n_ops]             integer cost, 1 <= cost <= 2^28; sum < 2^50
 *   op_input_offsets[n_ops+1]  CSR offsets into op_inputs (first 0, non-decreasing)
 *   op_inputs[...]             input tensor ids; each must be a constant or the
 *                              output of an earlier op; no duplicates per op
 * A tensor is released after the last op that reads it (after the op that
 * produces it, if nothing reads it), unless it is CONSTANT or REQUIRED.
 */
typedef struct {
    int32_t n_tensors, n_ops;
    const int64_t *tensor_size;
    const uint8_t *tensor_flags;
    const int32_t *op_output;
    const int64_t *op_cost;
    const int64_t *op_input_offsets;
    const int32_t *op_inputs;
} dtr_trace;

/* ---- deallocation policies: what releasing a tensor after its last reader
 * does (Section 2; Appendix C.4 and C.5; compared in Appendix D) ------------ */
#define DTR_POLICY_EAGER  0  /* evict it if resident, unlocked and not a constant   */
#define DTR_POLICY_IGNORE 1  /* nothing                                             */
#define DTR_POLICY_BANISH 2  /* if no child is evicted and no operation in progress
                                holds it: free it for good (constants included) and
                                pin its resident children (never evictable again);
                                else retry whenever one of its children is
                                rematerialized.  Not defined for the union-find
                                heuristics (DTR_H_EQ, DTR_C_EQCLASS): rejected.
                                Banishments are counted in n_eager_evictions. */

/* ---- search approximations of the prototype (Appendix E), bit flags ------ */
#define DTR_SEARCH_IGNORE_SMALL 1u  /* skip candidates with size below 1% of the
                                       pool's mean size (100 size n < sum)      */
#define DTR_SEARCH_SAMPLE       2u  /* search a random sample: each candidate kept
                                       with probability ceil(sqrt(n))/n, n = pool
                                       size, by a SplitMix64 draw per (seed ^
                                       0xD6E8FEB86659FD93, eviction number, id);
                                       if no candidate is left, every candidate
                                       that is not small is searched.  n_scores
                                       counts the candidates scored.            */

/* One simulation (32 bytes): trace index, DTR_H_* heuristic, memory budget
 * (same unit as tensor_size; DTR_BUDGET_UNLIMITED for none), seed (used by
 * DTR_H_RAND and DTR_SEARCH_SAMPLE), DTR_POLICY_* deallocation policy, and
 * DTR_SEARCH_* flags (0: exact search). */
typedef struct {
    int32_t trace;
    int32_t heuristic;
    int64_t budget;
    uint64_t seed;
    int32_t policy;
    int32_t search;
} dtr_sim_spec;

/* Result of one simulation (104 bytes). */
typedef struct {
    int64_t total_cost;        /* base_cost + remat_cost                                */
    int64_t base_cost;         /* cost of trace ops executed                            */
    int64_t remat_cost;        /* cost of rematerializations                            */
    int64_t peak_memory;       /* maximum memory in use                                 */
    int64_t final_memory;      /* memory in use when the run ended                      */
    int64_t n_executed_ops;    /* trace ops + rematerializations executed               */
    int64_t n_remats;          /* rematerializations                                    */
    int64_t n_evictions;       /* budget-driven evictions                               */
    int64_t n_eager_evictions; /* evictions on release                                  */
    int64_t n_scores;          /* candidates scored, summed over budget evictions       */
    int64_t n_nbr_visits;      /* h_DTR/h_ESTAR: sum of |e*|; h_EQ: evicted neighbours;
                                  summed over scored candidates; else 0                 */
    int64_t n_adj_visits;      /* h_DTR/h_EQ/h_ESTAR: sum of candidate degrees; else 0  */
    int32_t status;            /* DTR_STATUS_*                                          */
    int32_t failed_op;         /* op index being run when status != OK (n_ops while the
                                  output condition runs); -1 otherwise                  */
} dtr_sim_result;

/* Launch options (NULL = defaults). */
typedef struct {
    int32_t slots;   /* simulations resident on the GPU at once (0 = 16 per CU) */
    int32_t flags;   /* 0, or DTR_OPT_* bits                                    */
} dtr_sim_options;

/* Operator-log replay keeps every per-simulation array in device memory even
 * when the storage states, visited sets and storage graph of the batch's
 * largest log fit in LDS (results are identical; a testing aid).  Rejected
 * for traces. */
#define DTR_OPT_LOG_NO_LDS 1

/* Traces only, testing aids for the walk heuristics (h_DTR, h_{e*}, h_MSPS
 * and the family members with the e* cost): bits 8-11 set the wavefronts per
 * workgroup (1..8; 0 = chosen from the trace sizes), and
 * DTR_OPT_WALK_QUEUE_SMALL gives each lane a queue of 16 members, so that
 * larger neighbourhoods take the whole-wavefront walk.  Results are
 * identical either way. */
#define DTR_OPT_WALK_QUEUE_SMALL 4
#define DTR_OPT_WALK_WAVES_SHIFT 8
#define DTR_OPT_WALK_WAVES(w) ((w) << DTR_OPT_WALK_WAVES_SHIFT)

/* Traces only: the handle will run through dtr_sim_run_static, so its
 * workspace holds the inputs and results alone (no per-simulation working
 * memory); dtr_sim_run on it returns DTR_ESTATE.  Creation fails with
 * DTR_EINVAL if one simulation's working memory exceeds the static scratch. */
#define DTR_OPT_STATIC_SCRATCH 2

/* Size of the library's static device array used by dtr_sim_run_static. */
#define DTR_STATIC_SCRATCH_BYTES ((size_t)256 << 20)

typedef struct dtr_sim dtr_sim;

/* Device workspace size for this batch on the current device.  Validates the
 * traces and specs (DTR_ETRACE names the trace, op or sim and the reason). */
int dtr_sim_workspace_bytes(const dtr_trace *traces, int32_t n_traces,
                            const dtr_sim_spec *sims, int32_t n_sims,
                            const dtr_sim_options *options, size_t *bytes);

/* Validate, derive per-trace tables (producers, children, release lists),
 * lay out and upload everything into device_workspace on `stream`.  Host
 * arrays are copied; the caller may free them on return.  *out receives an
 * owned handle (free with dtr_sim_destroy). */
int dtr_sim_create(const dtr_trace *traces, int32_t n_traces,
                   const dtr_sim_spec *sims, int32_t n_sims,
                   const dtr_sim_options *options,
                   void *device_workspace, size_t workspace_bytes,
                   void *stream, dtr_sim **out);

/* Enqueue every simulation on `stream` (asynchronous, stream-ordered).  May be
 * called again; each call recomputes all results. */
int dtr_sim_run(dtr_sim *sim, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops): as dtr_sim_run, but every simulation's working
 * memory (state words, evictable pool, union-find nodes, rematerialization
 * stack, walk stamps and queues) and the work counters live in the
 * library's own static device array of DTR_STATIC_SCRATCH_BYTES, one per
 * device, held until the process ends, instead of in the handle's
 * workspace.  The inputs (uploaded by dtr_sim_create) and the results stay
 * in the handle's workspace; read them with dtr_sim_results.  As many
 * simulations are resident at once as the handle's slot count allows and
 * the array holds.  Allocates nothing and calls no allocating routine.
 * Errors: DTR_EINVAL for a NULL or operator-log handle, or when one
 * simulation's working memory exceeds the array; DTR_EHIP if a HIP call
 * fails.  Every call on a device shares that device's array and overwrites
 * it (the counters are cleared by a kernel at the start of each call):
 * calls that overlap in time on one device race, so order them (for
 * example on one stream). */
int dtr_sim_run_static(dtr_sim *sim, void *stream);

/* Copy n_sims results (== the batch size) into host_out, after synchronizing
 * the stream of the last run.  DTR_ESTATE if no run was enqueued. */
int dtr_sim_results(dtr_sim *sim, dtr_sim_result *host_out, int32_t n_sims);

/* Progress of the handle's last trace run, which may still be in flight:
 * the operations executed so far by its simulations under the e*-walking
 * heuristics (h_DTR, h_{e*}, h_MSPS and the h' members with c = e*), each
 * simulation counted in whole steps of 4096 operations (a lower bound; the
 * other heuristics and operator logs count 0).  It reads a device counter on
 * a stream of the handle's own (created at the first call), so it returns
 * without waiting for the run; for progress reports of long runs.
 * DTR_EINVAL for a NULL argument; *ops_done = 0 before any run. */
int dtr_sim_progress(dtr_sim *sim, int64_t *ops_done);

/* ---- operator logs (Appendix C.6) ------------------------------------------
 * A log is a sequence of instructions over integer names 0..n_names-1, as
 * parallel arrays (one entry per instruction):
 *   DTR_LOG_MEMORY    a = name, value = size in bytes (ignored for a view)
 *   DTR_LOG_ALIAS     a = name, b = the name it views, or -1 for a new storage
 *   DTR_LOG_CALL      ids[list_offsets[i] ..] = n_in input names, then the
 *                     output names (fresh); value = cost (1..2^28); each
 *                     output is then described by MEMORY and ALIAS, in output
 *                     order; a view must view an input or an earlier output of
 *                     the same call that owns a new storage
 *   DTR_LOG_MUTATE    ids = n_in input names, then the mutated ones (distinct,
 *                     among the inputs); value = cost.  Replayed as a pure
 *                     operator whose outputs are clones (new storages of the
 *                     same size); the mutated names are rebound to the clones
 *   DTR_LOG_CONSTANT  a = fresh name, then MEMORY: a nullary operator of cost 0
 *                     whose storage is pinned (never evicted)
 *   DTR_LOG_COPY      a = fresh name, b = name: one more reference to b's tensor
 *   DTR_LOG_COPYFROM  a = name rebound to b's tensor
 *   DTR_LOG_RELEASE   a = name dropped
 * Storages are the unit of eviction.  A storage whose references drop to zero
 * is released after the last operator issued (the deallocation policy then
 * applies); tensors still referenced at the end are required outputs.  A
 * tensor is defined when its storage is resident and its operator ran after
 * the storage last became resident; an operator call locks its inputs'
 * storages, defines undefined inputs in listed order, allocates every
 * non-view output, runs, frees the new copies of outputs that were already
 * defined, and unlocks (Appendix C.4).  A storage's cost sums the operator
 * cost of every tensor that views it, its dependencies are the storages those
 * operators read, its staleness counts from the latest reference to any of
 * its tensors (Appendix C.2).  Banishing a storage needs every tensor
 * computed from it (outside it) defined or gone, and pins their storages.
 * Results: operators count once per execution (views and constants
 * included); failed_op indexes operators in log order. */
#define DTR_LOG_MEMORY   0
#define DTR_LOG_ALIAS    1
#define DTR_LOG_CALL     2
#define DTR_LOG_MUTATE   3
#define DTR_LOG_CONSTANT 4
#define DTR_LOG_COPY     5
#define DTR_LOG_COPYFROM 6
#define DTR_LOG_RELEASE  7

typedef struct {
    int32_t n_instrs;
    int32_t n_names;
    const int32_t *kind;          /* [n_instrs] DTR_LOG_*                         */
    const int32_t *a;             /* [n_instrs] name operand                      */
    const int32_t *b;             /* [n_instrs] second name operand, or -1        */
    const int32_t *n_in;          /* [n_instrs] inputs in the list (CALL, MUTATE) */
    const int64_t *value;         /* [n_instrs] size (MEMORY) or cost             */
    const int64_t *list_offsets;  /* [n_instrs + 1] into ids                      */
    const int32_t *ids;           /* [list_offsets[n_instrs]]                     */
} dtr_log;

/* As dtr_sim_workspace_bytes / dtr_sim_create, for operator logs: the spec's
 * trace field indexes `logs`.  Logs are validated and lowered on the host
 * (DTR_ETRACE names the log, instruction and reason).  The handle is run,
 * read and destroyed with the dtr_sim_* calls below.  Every heuristic, policy
 * and search flag is accepted under the same rules as traces. */
int dtr_log_workspace_bytes(const dtr_log *logs, int32_t n_logs,
                            const dtr_sim_spec *sims, int32_t n_sims,
                            const dtr_sim_options *options, size_t *bytes);
int dtr_log_create(const dtr_log *logs, int32_t n_logs,
                   const dtr_sim_spec *sims, int32_t n_sims,
                   const dtr_sim_options *options,
                   void *device_workspace, size_t workspace_bytes,
                   void *stream, dtr_sim **out);

/* How a handle's simulations occupy the device, fixed at creation:
 * n_slots          simulations that can be in flight (one workgroup each,
 *                  except under exact h_DTR^eq: one wavefront each);
 * waves_per_group  wavefronts per workgroup: 1, except for operator logs
 *                  whose walk state is in LDS (up to 4) and for traces with
 *                  walk heuristics (up to 8): the first simulates, the
 *                  others join its e* / e_R walk scans; else 4 for traces
 *                  with exact h_DTR^eq simulations (a simulation per
 *                  wavefront);
 * lds_bytes        dynamic LDS per workgroup (0: the kernels' static LDS only,
 *                  or walk state in device memory).
 * Returns DTR_EINVAL for a NULL argument.  No device work. */
typedef struct {
    int32_t n_slots;
    int32_t waves_per_group;
    int32_t lds_bytes;
    int32_t reserved;            /* 0 */
} dtr_launch_info;

int dtr_sim_launch_info(const dtr_sim *sim, dtr_launch_info *out);

/* Release the handle (not the caller's workspace).  NULL is ignored. */
void dtr_sim_destroy(dtr_sim *sim);

/* Message of the last failing call on this thread ("" if none). */
const char *dtr_sim_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DTR_SIM_H */
