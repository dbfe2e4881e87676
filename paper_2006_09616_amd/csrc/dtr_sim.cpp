// dtr_sim.cpp -- host side of the C ABI declared in include/dtr_sim.h:
// validation, per-trace derivation, workspace layout, upload and launch.
//
// Derivation (once per trace, host): the parent operation of every tensor
// and its cost c0 (Appendix C.2 "Cost"), children (the dependents deps^T of
// Appendix C.2 "Data dependencies"), the undirected neighbourhood used by the
// union-find relaxation, the release point of every tensor (after its last
// reader, from reference counting as in Appendix A.2 "Liveness"), required
// outputs and constants.  All tables are uploaded once into the caller's
// device workspace and shared read-only by every simulation of the trace.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <numeric>
#include <string>
#include <vector>

#include "../../include/dtr_sim.h"
#include "host.h"
#include "layout.h"

extern "C" hipError_t dtr_launch_reset(uint32_t *queue, hipStream_t stream);
extern "C" hipError_t dtr_launch_group(const dtr::KernelArgs *a, int32_t group, hipStream_t stream);
extern "C" hipError_t dtr_static_scratch(void **ptr, size_t *bytes);

namespace dtrhost {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

bool heuristic_known(int32_t h)
{
    return (h >= DTR_H_DTR && h <= DTR_H_MSPS) || (h >= DTR_H_FAMILY(0, 0, 0) && h <= DTR_H_FAMILY(3, 1, 1));
}

int32_t heuristic_class(int32_t h)
{
    if (h >= DTR_H_FAMILY(0, 0, 0)) {
        const int32_t c = (h - DTR_H_FAMILY(0, 0, 0)) >> 2;
        return c == DTR_C_EQCLASS ? 0 : c == DTR_C_ESTAR ? 1 : 2;
    }
    return h == DTR_H_EQ ? 0 : (h == DTR_H_DTR || h == DTR_H_ESTAR || h == DTR_H_MSPS) ? 1 : 2;
}

int check_spec(const dtr_sim_spec &s, int32_t i)
{
    if (!heuristic_known(s.heuristic)) return fail(DTR_ETRACE, "sim %d: unknown heuristic %d", i, s.heuristic);
    if (s.budget < 0) return fail(DTR_ETRACE, "sim %d: negative budget", i);
    if (s.policy < DTR_POLICY_EAGER || s.policy > DTR_POLICY_BANISH)
        return fail(DTR_ETRACE, "sim %d: unknown deallocation policy %d", i, s.policy);
    if (s.policy == DTR_POLICY_BANISH && heuristic_class(s.heuristic) == 0)
        return fail(DTR_ETRACE, "sim %d: banishing is not defined for union-find heuristics", i);
    if (s.search & ~(int32_t)(DTR_SEARCH_IGNORE_SMALL | DTR_SEARCH_SAMPLE))
        return fail(DTR_ETRACE, "sim %d: unknown search flags %d", i, s.search);
    return DTR_OK;
}

int device_cus(int32_t *cus)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(DTR_EHIP, "hipGetDevice failed");
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return fail(DTR_EHIP, "hipDeviceGetAttribute(multiProcessorCount) failed");
    *cus = v;
    return DTR_OK;
}

}  // namespace dtrhost

namespace {

using namespace dtrhost;

// dtr_sim_run_static: work counters, then slots, in the static scratch
constexpr size_t STATIC_HEADER = 256;
constexpr int32_t MAX_TENSORS = 8000000;       // pool positions are packed in 24 bits
constexpr int32_t MAX_DEGREE = (1 << 23) - 1;  // degrees are packed in 23 bits

struct Derived {
    int32_t n = 0, F = 0;
    std::vector<int64_t> size, c0, cost;
    std::vector<uint8_t> flags;
    std::vector<int32_t> producer, out, in_off, in, ch_off, ch, adj_off, adj, rel_off, rel, req, consts;
    std::vector<dtr::TRecX> rec;
    int64_t const_mem = 0;
    int64_t peak = 0;        // memory with no eviction: frees at release points (dispatch order)
};

int validate_and_derive(const dtr_trace &tr, int32_t index, Derived &d)
{
    if (tr.n_tensors < 0 || tr.n_ops < 0)
        return fail(DTR_ETRACE, "trace %d: negative n_tensors or n_ops", index);
    if (tr.n_tensors > MAX_TENSORS)
        return fail(DTR_ETRACE, "trace %d: %d tensors exceed the limit of %d", index, tr.n_tensors, MAX_TENSORS);
    if ((tr.n_tensors > 0 && (!tr.tensor_size || !tr.tensor_flags)) ||
        (tr.n_ops > 0 && (!tr.op_output || !tr.op_cost || !tr.op_inputs)) || !tr.op_input_offsets)
        return fail(DTR_EINVAL, "trace %d: null array", index);
    const int32_t n = tr.n_tensors, F = tr.n_ops;
    d.n = n;
    d.F = F;
    d.size.assign(tr.tensor_size, tr.tensor_size + n);
    d.flags.assign(tr.tensor_flags, tr.tensor_flags + n);
    for (int32_t t = 0; t < n; t++) {
        if (d.size[t] < 1 || d.size[t] >= MAX_SIZE)
            return fail(DTR_ETRACE, "trace %d: tensor %d size %lld outside [1, 2^36)", index, t,
                        (long long)d.size[t]);
        if (d.flags[t] & ~(DTR_FLAG_CONSTANT | DTR_FLAG_REQUIRED))
            return fail(DTR_ETRACE, "trace %d: tensor %d has unknown flag bits", index, t);
    }
    if (tr.op_input_offsets[0] != 0) return fail(DTR_ETRACE, "trace %d: op_input_offsets[0] != 0", index);
    const int64_t E = tr.op_input_offsets[F];
    if (E < 0 || E > (int64_t(1) << 30)) return fail(DTR_ETRACE, "trace %d: %lld edges", index, (long long)E);
    d.producer.assign(n, -1);
    d.c0.assign(n, 0);
    d.out.assign(tr.op_output, tr.op_output + F);
    d.cost.assign(tr.op_cost, tr.op_cost + F);
    d.in_off.resize(F + 1);
    d.in.resize(E);
    std::vector<uint8_t> defined(n, 0);
    std::vector<int32_t> seen(n, -1);
    for (int32_t t = 0; t < n; t++) defined[t] = (d.flags[t] & DTR_FLAG_CONSTANT) ? 1 : 0;
    int64_t total = 0;
    std::vector<int32_t> last(n, -1);
    for (int32_t o = 0; o < F; o++) {
        const int64_t b = tr.op_input_offsets[o], e = tr.op_input_offsets[o + 1];
        if (e < b || e > E) return fail(DTR_ETRACE, "trace %d: op %d: offsets not monotone", index, o);
        const int64_t c = d.cost[o];
        if (c < 1 || c > MAX_COST)
            return fail(DTR_ETRACE, "trace %d: op %d: cost %lld outside [1, 2^28]", index, o, (long long)c);
        total += c;
        if (total >= MAX_TOTAL_COST) return fail(DTR_ETRACE, "trace %d: total cost reaches 2^50", index);
        d.in_off[o] = (int32_t)b;
        for (int64_t k = b; k < e; k++) {
            const int32_t u = tr.op_inputs[k];
            if (u < 0 || u >= n) return fail(DTR_ETRACE, "trace %d: op %d: input %d out of range", index, o, u);
            if (!defined[u])
                return fail(DTR_ETRACE, "trace %d: op %d: input %d is not defined before use", index, o, u);
            if (seen[u] == o) return fail(DTR_ETRACE, "trace %d: op %d: duplicate input %d", index, o, u);
            seen[u] = o;
            d.in[k] = u;
            last[u] = o;
        }
        const int32_t t = d.out[o];
        if (t < 0 || t >= n) return fail(DTR_ETRACE, "trace %d: op %d: output %d out of range", index, o, t);
        if (defined[t])
            return fail(DTR_ETRACE, "trace %d: op %d: tensor %d is a constant or already produced", index, o, t);
        defined[t] = 1;
        d.producer[t] = o;
        d.c0[t] = c;
        if (last[t] < o) last[t] = o;
    }
    d.in_off[F] = (int32_t)E;
    for (int32_t t = 0; t < n; t++)
        if (!defined[t]) return fail(DTR_ETRACE, "trace %d: tensor %d is never produced", index, t);

    // children CSR (ascending consumer op order)
    d.ch_off.assign(n + 1, 0);
    for (int64_t k = 0; k < E; k++) d.ch_off[d.in[k] + 1]++;
    for (int32_t t = 0; t < n; t++) d.ch_off[t + 1] += d.ch_off[t];
    d.ch.resize(E);
    {
        std::vector<int32_t> fill(d.ch_off.begin(), d.ch_off.end() - 1);
        for (int32_t o = 0; o < F; o++)
            for (int32_t k = d.in_off[o]; k < d.in_off[o + 1]; k++) d.ch[fill[d.in[k]]++] = d.out[o];
    }
    // undirected neighbourhood: parents then children
    d.adj_off.assign(n + 1, 0);
    for (int32_t t = 0; t < n; t++) {
        const int32_t o = d.producer[t];
        const int32_t np = o >= 0 ? d.in_off[o + 1] - d.in_off[o] : 0;
        d.adj_off[t + 1] = d.adj_off[t] + np + (d.ch_off[t + 1] - d.ch_off[t]);
    }
    for (int32_t t = 0; t < n; t++)
        if (d.adj_off[t + 1] - d.adj_off[t] > MAX_DEGREE)
            return fail(DTR_ETRACE, "trace %d: tensor %d has more than %d neighbours", index, t, MAX_DEGREE);
    d.adj.resize(d.adj_off[n]);
    for (int32_t t = 0; t < n; t++) {
        int32_t w = d.adj_off[t];
        const int32_t o = d.producer[t];
        if (o >= 0)
            for (int32_t k = d.in_off[o]; k < d.in_off[o + 1]; k++) d.adj[w++] = d.in[k];
        for (int32_t k = d.ch_off[t]; k < d.ch_off[t + 1]; k++) d.adj[w++] = d.ch[k];
    }
    // release lists, ascending id
    d.rel_off.assign(F + 1, 0);
    for (int32_t t = 0; t < n; t++)
        if (!(d.flags[t] & DTR_FLAG_REQUIRED) && last[t] >= 0) d.rel_off[last[t] + 1]++;
    for (int32_t o = 0; o < F; o++) d.rel_off[o + 1] += d.rel_off[o];
    d.rel.resize(d.rel_off[F]);
    {
        std::vector<int32_t> fill(d.rel_off.begin(), d.rel_off.end() - 1);
        for (int32_t t = 0; t < n; t++)
            if (!(d.flags[t] & DTR_FLAG_REQUIRED) && last[t] >= 0) d.rel[fill[last[t]]++] = t;
    }
    {
        int64_t mem = 0;
        for (int32_t t = 0; t < n; t++)
            if (d.flags[t] & DTR_FLAG_CONSTANT) mem += d.size[t];
        d.peak = mem;
        for (int32_t o = 0; o < F; o++) {
            mem += d.size[d.out[o]];
            d.peak = std::max(d.peak, mem);
            for (int32_t k = d.rel_off[o]; k < d.rel_off[o + 1]; k++)
                if (!(d.flags[d.rel[k]] & DTR_FLAG_CONSTANT)) mem -= d.size[d.rel[k]];
        }
    }
    d.rec.resize(n);
    for (int32_t t = 0; t < n; t++) {
        dtr::TRec &r = d.rec[t].r;
        const int32_t o = d.producer[t];
        r.size = d.size[t];
        r.c0 = (int32_t)d.c0[t];
        r.producer = o;
        r.in_b = o >= 0 ? d.in_off[o] : 0;
        r.in_e = o >= 0 ? d.in_off[o + 1] : 0;
        r.adj_b = d.adj_off[t];
        r.adj_e = d.adj_off[t + 1];
        for (int32_t j = 0; j < dtr::NB_HEAD; j++)
            d.rec[t].nb[j] = d.adj_off[t] + j < d.adj_off[t + 1] ? d.adj[d.adj_off[t] + j] : 0;
    }
    for (int32_t t = 0; t < n; t++) {
        if (d.flags[t] & DTR_FLAG_REQUIRED) d.req.push_back(t);
        if (d.flags[t] & DTR_FLAG_CONSTANT) {
            d.consts.push_back(t);
            d.const_mem += d.size[t];
        }
    }
    return DTR_OK;
}

// workspace: [header | trace tables | trace descriptors | specs | order | results | slots]
struct Plan {
    std::vector<Derived> traces;
    std::vector<size_t> trace_off;   // start of each trace's tables
    size_t desc_off = 0, spec_off = 0, order_off = 0, result_off = 0, slot_off = 0, prof_off = 0;
    size_t tables_bytes = 0;         // everything before the slots (uploaded)
    size_t total = 0;
    dtr::SlotLayout L{};
    int32_t n_slots = 0;
    bool static_only = false;        // runs only through dtr_sim_run_static: no slots in the workspace
    std::vector<int32_t> order;
    int32_t class_count[dtr::N_GROUPS] = {0, 0, 0, 0, 0, 0};
};

template <class T>
size_t bytes_of(const std::vector<T> &v) { return align_up(v.size() * sizeof(T)); }

size_t trace_bytes(const Derived &d)
{
    return bytes_of(d.size) + bytes_of(d.c0) + bytes_of(d.flags) + bytes_of(d.producer) + bytes_of(d.out) +
           bytes_of(d.cost) + bytes_of(d.in_off) + bytes_of(d.in) + bytes_of(d.ch_off) + bytes_of(d.ch) +
           bytes_of(d.adj_off) + bytes_of(d.adj) + bytes_of(d.rel_off) + bytes_of(d.rel) + bytes_of(d.req) +
           bytes_of(d.consts) + bytes_of(d.rec) + 8 * ALIGN;
}

int make_plan(const dtr_trace *traces, int32_t n_traces, const dtr_sim_spec *sims, int32_t n_sims,
              const dtr_sim_options *opt, Plan &p)
{
    if (n_traces < 0 || n_sims < 0) return fail(DTR_EINVAL, "negative n_traces or n_sims");
    if ((n_traces > 0 && !traces) || (n_sims > 0 && !sims)) return fail(DTR_EINVAL, "null traces or sims");
    if (opt && (opt->slots < 0 || (opt->flags & ~(DTR_OPT_STATIC_SCRATCH | DTR_OPT_WALK_QUEUE_SMALL |
                                                  (15 << DTR_OPT_WALK_WAVES_SHIFT)))))
        return fail(DTR_EINVAL, "bad options");
    if (opt && ((opt->flags >> DTR_OPT_WALK_WAVES_SHIFT) & 15) > dtr::MAX_WALK_WAVES)
        return fail(DTR_EINVAL, "at most %d wavefronts per walk workgroup", dtr::MAX_WALK_WAVES);
    p.static_only = opt && (opt->flags & DTR_OPT_STATIC_SCRATCH);
    p.traces.resize(n_traces);
    for (int32_t i = 0; i < n_traces; i++) {
        int rc = validate_and_derive(traces[i], i, p.traces[i]);
        if (rc) return rc;
    }
    bool need_uf = false, need_walk = false, need_banish = false;
    int32_t n_max = 1;
    for (int32_t i = 0; i < n_sims; i++) {
        const dtr_sim_spec &s = sims[i];
        if (s.trace < 0 || s.trace >= n_traces)
            return fail(DTR_ETRACE, "sim %d: trace index %d out of range", i, s.trace);
        if (int rc = check_spec(s, i)) return rc;
        need_banish |= s.policy == DTR_POLICY_BANISH;
        need_uf |= heuristic_class(s.heuristic) == 0;
        need_walk |= heuristic_class(s.heuristic) == 1;
        n_max = std::max(n_max, p.traces[s.trace].n);
    }
    // slot layout
    dtr::SlotLayout &L = p.L;
    size_t o = 0;
    auto take = [&](int64_t &field, size_t bytes) { field = (int64_t)o; o += align_up(bytes); };
    const size_t n = (size_t)n_max;
    L.n_max = n_max;
    L.pcap = 2 * (int64_t)n + 128;
    L.ucap = need_uf ? 2 * (int64_t)n + 64 : 0;
    const size_t pc = (size_t)L.pcap;
    take(L.tst, 8 * n);
    take(L.lockx, 4 * n);
    take(L.pool, sizeof(dtr::PoolSlot) * pc);
    take(L.nodes, sizeof(dtr::UfNode) * (size_t)L.ucap);
    take(L.uf_remap, need_uf ? 4 * ((size_t)L.ucap + dtr::UF_LDS) : 0);
    take(L.stack, sizeof(dtr::StackFrame) * (size_t)(n + 1));
    // walk heuristics: wavefronts per workgroup (more for large traces, whose
    // pools are long), a visited bitmap and a member queue per lane
    int32_t ww = opt ? (opt->flags >> DTR_OPT_WALK_WAVES_SHIFT) & 15 : 0;
    if (ww == 0) ww = n_max >= 8192 ? dtr::MAX_WALK_WAVES : n_max >= 1024 ? 4 : 1;
    L.walk_waves = need_walk ? ww : 1;
    const size_t lanes = (size_t)L.walk_waves * dtr::WAVE;
    L.vis_words = (int64_t)((n + 127) / 128 * 4);
    L.vis_bytes = (int64_t)((n + 15) / 16 * 16);
    L.wq_cap = (opt && (opt->flags & DTR_OPT_WALK_QUEUE_SMALL)) ? 16
                                                                  : std::min<int64_t>((int64_t)n + 1, dtr::WALK_QUEUE_CAP);
    take(L.vis, need_walk ? (size_t)L.vis_bytes * lanes : 0);
    take(L.wq, need_walk ? 4 * (size_t)L.wq_cap * lanes : 0);
    take(L.bigvis, need_walk ? 4 * (size_t)L.vis_words * (size_t)L.walk_waves : 0);
    take(L.bigq, need_walk ? 4 * (n + 1) * (size_t)L.walk_waves : 0);
    take(L.ovf, need_walk ? 4 * pc : 0);
    take(L.pending, need_banish ? n : 0);
    L.bytes = (int64_t)o;
    if (p.static_only && (size_t)L.bytes > DTR_STATIC_SCRATCH_BYTES - STATIC_HEADER)
        return fail(DTR_EINVAL, "one simulation needs %lld bytes of working memory; the static scratch holds %zu",
                    (long long)L.bytes, (size_t)(DTR_STATIC_SCRATCH_BYTES - STATIC_HEADER));

    int32_t cus = 0;
    int rc = device_cus(&cus);
    if (rc) return rc;
    // 16 slots per compute unit (at least as many as any kernel keeps
    // resident: 8 under h_DTR^eq, one per wavefront); a batch of walk
    // heuristics alone needs no more slots than its larger workgroups occupy
    const bool walk_only = need_walk && !need_uf && [&] {
        for (int32_t i = 0; i < n_sims; i++)
            if (heuristic_class(sims[i].heuristic) != 1) return false;
        return true;
    }();
    int64_t slots = opt && opt->slots > 0 ? opt->slots
                                          : (int64_t)cus * (walk_only ? std::max<int64_t>(1, 16 / L.walk_waves) : 16);
    const int64_t cap_bytes = int64_t(48) << 30;     // bound slot memory
    slots = std::min<int64_t>(slots, std::max<int64_t>(1, cap_bytes / std::max<int64_t>(1, L.bytes)));
    slots = std::min<int64_t>(slots, std::max<int32_t>(1, n_sims));
    p.n_slots = (int32_t)std::max<int64_t>(1, slots);

    // grouped by heuristic class (one kernel specialisation each), then the
    // Likely heaviest first: each trace's tightest simulation (budget relative
    // to the trace's no-eviction peak, in steps of 1/1024 of the peak, so
    // that budgets set at one fraction of their traces' peaks tie) before the
    // rest, those by tightness, then the longest trace, then the exact ratio;
    // then the rest trace by trace (longest first), each trace's tightest
    // first, so that the simulations of one trace run side by side and share
    // its tables in the caches.
    auto cls = [&](int32_t i) { return heuristic_class(sims[i].heuristic) + (sims[i].search ? 3 : 0); };
    auto bucket = [&](int32_t i) {
        const uint64_t pk = (uint64_t)std::max<int64_t>(1, p.traces[sims[i].trace].peak);
        return (unsigned __int128)(uint64_t)sims[i].budget * 1024u / pk;
    };
    std::map<std::pair<int32_t, int32_t>, unsigned __int128> tightest;     // (trace, group) -> bucket
    for (int32_t i = 0; i < n_sims; i++) {
        const auto key = std::make_pair(sims[i].trace, cls(i));
        const auto it = tightest.find(key);
        if (it == tightest.end() || bucket(i) < it->second) tightest[key] = bucket(i);
    }
    std::vector<uint8_t> first(n_sims);
    for (int32_t i = 0; i < n_sims; i++) first[i] = bucket(i) == tightest[std::make_pair(sims[i].trace, cls(i))];
    p.order.resize(n_sims);
    std::iota(p.order.begin(), p.order.end(), 0);
    std::stable_sort(p.order.begin(), p.order.end(), [&](int32_t a, int32_t b) {
        if (cls(a) != cls(b)) return cls(a) < cls(b);
        if (first[a] != first[b]) return first[a] > first[b];
        const Derived &ta = p.traces[sims[a].trace], &tb = p.traces[sims[b].trace];
        if (!first[a]) {
            if (ta.F != tb.F) return ta.F > tb.F;
            if (sims[a].trace != sims[b].trace) return sims[a].trace < sims[b].trace;
        }
        const uint64_t pa = (uint64_t)std::max<int64_t>(1, ta.peak), pb = (uint64_t)std::max<int64_t>(1, tb.peak);
        const unsigned __int128 qa = (unsigned __int128)(uint64_t)sims[a].budget * 1024u / pa;
        const unsigned __int128 qb = (unsigned __int128)(uint64_t)sims[b].budget * 1024u / pb;
        if (qa != qb) return qa < qb;
        if (ta.F != tb.F) return ta.F > tb.F;
        const unsigned __int128 ra = (unsigned __int128)(uint64_t)sims[a].budget * pb;
        const unsigned __int128 rb = (unsigned __int128)(uint64_t)sims[b].budget * pa;
        if (ra != rb) return ra < rb;
        return sims[a].budget < sims[b].budget;
    });
    for (int c = 0; c < dtr::N_GROUPS; c++) p.class_count[c] = 0;
    for (int32_t i = 0; i < n_sims; i++) p.class_count[cls(i)]++;

    size_t w = align_up(64);   // header: work counter
    p.trace_off.resize(n_traces);
    for (int32_t i = 0; i < n_traces; i++) {
        p.trace_off[i] = w;
        w += trace_bytes(p.traces[i]);
    }
    p.desc_off = w;
    w += align_up(sizeof(dtr::TraceDev) * std::max(1, n_traces));
    p.spec_off = w;
    w += align_up(sizeof(dtr::SpecDev) * std::max(1, n_sims));
    p.order_off = w;
    w += align_up(sizeof(int32_t) * std::max(1, n_sims));
    p.tables_bytes = w;
    p.result_off = w;
    w += align_up(sizeof(dtr::ResultDev) * std::max(1, n_sims));
#ifdef DTR_PROFILE
    p.prof_off = w;
    w += align_up(sizeof(int64_t) * dtr::PROF_FIELDS * std::max(1, n_sims));
#endif
    p.slot_off = w;
    if (!p.static_only) w += (size_t)L.bytes * (size_t)p.n_slots;
    p.total = w;
    return DTR_OK;
}

}  // namespace

struct dtr_sim {
    Plan plan;
    dtrhost::LogPlan *log = nullptr;    // set for operator logs
    uint8_t *ws = nullptr;
    size_t ws_bytes = 0;
    std::vector<uint8_t> staging;
    hipStream_t last_stream = nullptr;
    bool ran = false;
    int32_t n_sims = 0;
    // a batch with simulations in several groups runs each group's kernel on
    // a stream of its own (default priority), forked from and joined back to
    // the caller's stream by events, so that the groups overlap
    hipStream_t aux[dtr::N_GROUPS] = {};
    hipEvent_t fork = nullptr, join[dtr::N_GROUPS] = {};
    uint32_t *last_queue = nullptr;       // counter block of the last trace run
    hipStream_t progress_stream = nullptr;  // dtr_sim_progress's reads
    ~dtr_sim()
    {
        dtrhost::log_plan_free(log);
        for (int g = 0; g < dtr::N_GROUPS; g++) {
            if (aux[g]) (void)hipStreamDestroy(aux[g]);
            if (join[g]) (void)hipEventDestroy(join[g]);
        }
        if (fork) (void)hipEventDestroy(fork);
        if (progress_stream) (void)hipStreamDestroy(progress_stream);
    }
};

extern "C" {

const char *dtr_sim_last_error(void) { return g_err.c_str(); }

int dtr_sim_workspace_bytes(const dtr_trace *traces, int32_t n_traces, const dtr_sim_spec *sims, int32_t n_sims,
                            const dtr_sim_options *options, size_t *bytes)
{
    g_err.clear();
    if (!bytes) return fail(DTR_EINVAL, "null bytes");
    Plan p;
    int rc = make_plan(traces, n_traces, sims, n_sims, options, p);
    if (rc) return rc;
    *bytes = p.total;
    return DTR_OK;
}

int dtr_sim_create(const dtr_trace *traces, int32_t n_traces, const dtr_sim_spec *sims, int32_t n_sims,
                   const dtr_sim_options *options, void *device_workspace, size_t workspace_bytes, void *stream,
                   dtr_sim **out)
{
    g_err.clear();
    if (!out) return fail(DTR_EINVAL, "null out");
    *out = nullptr;
    if (!device_workspace) return fail(DTR_EINVAL, "null device workspace");
    if ((uintptr_t)device_workspace % ALIGN) return fail(DTR_EINVAL, "workspace must be 256-byte aligned");
    dtr_sim *h = new dtr_sim();
    int rc = make_plan(traces, n_traces, sims, n_sims, options, h->plan);
    if (rc) { delete h; return rc; }
    Plan &p = h->plan;
    if (workspace_bytes < p.total) {
        rc = fail(DTR_EINVAL, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, p.total);
        delete h;
        return rc;
    }
    h->ws = (uint8_t *)device_workspace;
    h->ws_bytes = workspace_bytes;
    h->n_sims = n_sims;
    h->staging.assign(p.tables_bytes, 0);
    uint8_t *H = h->staging.data();
    std::vector<dtr::TraceDev> descs(std::max(1, n_traces));
    for (int32_t i = 0; i < n_traces; i++) {
        const Derived &d = p.traces[i];
        size_t w = p.trace_off[i];
        auto put = [&](const auto &v) {
            using T = typename std::decay_t<decltype(v)>::value_type;
            size_t at = w;
            if (!v.empty()) std::memcpy(H + at, v.data(), v.size() * sizeof(T));
            w += bytes_of(v);
            return (const T *)(h->ws + at);
        };
        dtr::TraceDev &D = descs[i];
        D.n = d.n;
        D.F = d.F;
        D.n_req = (int32_t)d.req.size();
        D.n_const = (int32_t)d.consts.size();
        D.const_mem = d.const_mem;
        D.size = put(d.size);
        D.c0 = put(d.c0);
        D.flags = put(d.flags);
        D.producer = put(d.producer);
        D.out = put(d.out);
        D.cost = put(d.cost);
        D.in_off = put(d.in_off);
        D.in = put(d.in);
        D.ch_off = put(d.ch_off);
        D.ch = put(d.ch);
        D.adj_off = put(d.adj_off);
        D.adj = put(d.adj);
        D.rel_off = put(d.rel_off);
        D.rel = put(d.rel);
        D.req = put(d.req);
        D.consts = put(d.consts);
        D.rec = put(d.rec);
    }
    std::memcpy(H + p.desc_off, descs.data(), sizeof(dtr::TraceDev) * n_traces);
    for (int32_t i = 0; i < n_sims; i++) {
        dtr::SpecDev s{sims[i].trace, sims[i].heuristic, sims[i].budget, sims[i].seed, sims[i].policy,
                       sims[i].search};
        std::memcpy(H + p.spec_off + i * sizeof(dtr::SpecDev), &s, sizeof(s));
    }
    if (n_sims) std::memcpy(H + p.order_off, p.order.data(), sizeof(int32_t) * n_sims);
    hipStream_t st = (hipStream_t)stream;
    int groups = 0;
    for (int c = 0; c < dtr::N_GROUPS; c++) groups += p.class_count[c] > 0;
    if (groups > 1) {
        bool okk = hipEventCreateWithFlags(&h->fork, hipEventDisableTiming) == hipSuccess;
        for (int c = 0; okk && c < dtr::N_GROUPS; c++)
            if (p.class_count[c] > 0)
                okk = hipStreamCreateWithFlags(&h->aux[c], hipStreamNonBlocking) == hipSuccess &&
                      hipEventCreateWithFlags(&h->join[c], hipEventDisableTiming) == hipSuccess;
        if (!okk) {
            rc = fail(DTR_EHIP, "stream or event creation failed");
            delete h;
            return rc;
        }
    }
    if (hipMemcpyAsync(h->ws, H, p.tables_bytes, hipMemcpyHostToDevice, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess) {
        rc = fail(DTR_EHIP, "upload of %zu bytes failed", p.tables_bytes);
        delete h;
        return rc;
    }
    *out = h;
    return DTR_OK;
}

}  // extern "C"

namespace {

// Enqueue the replay kernels of a trace batch: slots from `slots` (at most
// `max_slots` resident simulations), work counters at `queue`.  When several
// groups have simulations, the slots are shared out in proportion to their
// simulations and each group's kernel runs on its own stream.
int launch_traces(dtr_sim *h, void *stream, uint8_t *slots, uint32_t *queue, int64_t max_slots)
{
    const Plan &p = h->plan;
    hipStream_t st = (hipStream_t)stream;
    const int64_t total = std::max<int64_t>(1, std::min<int64_t>(p.n_slots, max_slots));
    int32_t groups[dtr::N_GROUPS], ng = 0;
    for (int c = 0; c < dtr::N_GROUPS; c++)
        if (p.class_count[c] > 0) groups[ng++] = c;
    // concurrent groups take disjoint slot ranges, each at least one slot;
    // with fewer slots than groups the groups run one after another on the
    // caller's stream, each over every slot
    const bool fan = ng > 1 && h->fork && total >= ng;
    int64_t share[dtr::N_GROUPS] = {0, 0, 0, 0, 0, 0};
    for (int k = 0; k < ng; k++) {
        const int c = groups[k];
        share[c] = !fan ? total : std::max<int64_t>(1, total * p.class_count[c] / std::max(1, h->n_sims));
        share[c] = std::min<int64_t>(share[c], p.class_count[c]);
    }
    for (; fan;) {      // trim the largest shares until the ranges fit
        int64_t sum = 0;
        int big = -1;
        for (int k = 0; k < ng; k++) {
            sum += share[groups[k]];
            if (share[groups[k]] > 1 && (big < 0 || share[groups[k]] > share[big])) big = groups[k];
        }
        if (sum <= total) break;
        share[big]--;
    }
    dtr::KernelArgs a[dtr::N_GROUPS];
    int32_t first = 0;
    int64_t off = 0;
    for (int c = 0; c < dtr::N_GROUPS; c++) {
        a[c].traces = (const dtr::TraceDev *)(h->ws + p.desc_off);
        a[c].specs = (const dtr::SpecDev *)(h->ws + p.spec_off);
        a[c].order = (const int32_t *)(h->ws + p.order_off) + first;
        a[c].results = (dtr::ResultDev *)(h->ws + p.result_off);
        a[c].queue = queue + c;
        a[c].progress = (unsigned long long *)((uint8_t *)queue + dtr::PROGRESS_OFFSET);
        a[c].slots = slots + (size_t)off * (size_t)p.L.bytes;
        a[c].L = p.L;
        a[c].n_sims = p.class_count[c];
        a[c].n_slots = (int32_t)std::max<int64_t>(1, share[c]);
        a[c].prof = nullptr;
#ifdef DTR_PROFILE
        a[c].prof = (int64_t *)(h->ws + p.prof_off);
#endif
        first += p.class_count[c];
        if (fan) off += share[c];
    }
    hipError_t e = dtr_launch_reset(queue, st);
    if (e == hipSuccess && fan) e = hipEventRecord(h->fork, st);
    for (int k = 0; e == hipSuccess && k < ng; k++) {
        const int c = groups[k];
        hipStream_t gs = fan && k > 0 ? h->aux[c] : st;
        if (gs != st) e = hipStreamWaitEvent(gs, h->fork, 0);
        if (e == hipSuccess) e = dtr_launch_group(&a[c], c, gs);
        if (e == hipSuccess && gs != st) e = hipEventRecord(h->join[c], gs);
        if (e == hipSuccess && gs != st) e = hipStreamWaitEvent(st, h->join[c], 0);
    }
    if (e != hipSuccess) return fail(DTR_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    h->ran = true;
    h->last_stream = st;
    h->last_queue = queue;
    return DTR_OK;
}

}  // namespace

extern "C" {

int dtr_sim_run(dtr_sim *h, void *stream)
{
    g_err.clear();
    if (!h) return fail(DTR_EINVAL, "null handle");
    const Plan &p = h->plan;
    if (h->n_sims == 0) { h->ran = true; h->last_stream = (hipStream_t)stream; return DTR_OK; }
    if (h->log) {
        if (int rc = dtrhost::log_plan_launch(h->log, h->ws, (hipStream_t)stream)) return rc;
        h->ran = true;
        h->last_stream = (hipStream_t)stream;
        return DTR_OK;
    }
    if (p.static_only)
        return fail(DTR_ESTATE, "the handle was created with DTR_OPT_STATIC_SCRATCH: run it with dtr_sim_run_static");
    return launch_traces(h, stream, h->ws + p.slot_off, (uint32_t *)h->ws, p.n_slots);
}

int dtr_sim_run_static(dtr_sim *h, void *stream)
{
    g_err.clear();
    if (!h) return fail(DTR_EINVAL, "null handle");
    if (h->log) return fail(DTR_EINVAL, "dtr_sim_run_static runs traces only");
    const Plan &p = h->plan;
    if (h->n_sims == 0) { h->ran = true; h->last_stream = (hipStream_t)stream; return DTR_OK; }
    void *base = nullptr;
    size_t cap = 0;
    const hipError_t e = dtr_static_scratch(&base, &cap);
    if (e != hipSuccess) return fail(DTR_EHIP, "static scratch lookup failed: %s", hipGetErrorString(e));
    if ((size_t)p.L.bytes > cap - STATIC_HEADER)
        return fail(DTR_EINVAL, "one simulation needs %lld bytes of working memory; the static scratch holds %zu",
                    (long long)p.L.bytes, cap - STATIC_HEADER);
    const int64_t fit = (int64_t)((cap - STATIC_HEADER) / (size_t)p.L.bytes);
    return launch_traces(h, stream, (uint8_t *)base + STATIC_HEADER, (uint32_t *)base, fit);
}

int dtr_sim_results(dtr_sim *h, dtr_sim_result *host_out, int32_t n_sims)
{
    g_err.clear();
    if (!h || (!host_out && n_sims > 0)) return fail(DTR_EINVAL, "null handle or output");
    if (n_sims != h->n_sims) return fail(DTR_EINVAL, "n_sims %d does not match the batch (%d)", n_sims, h->n_sims);
    if (!h->ran) return fail(DTR_ESTATE, "no run enqueued");
    if (n_sims == 0) return DTR_OK;
    static_assert(sizeof(dtr_sim_result) == sizeof(dtr::ResultDev), "result layout");
    const size_t result_off = h->log ? dtrhost::log_plan_result_off(h->log) : h->plan.result_off;
    if (hipMemcpyAsync(host_out, h->ws + result_off, sizeof(dtr_sim_result) * n_sims,
                       hipMemcpyDeviceToHost, h->last_stream) != hipSuccess ||
        hipStreamSynchronize(h->last_stream) != hipSuccess)
        return fail(DTR_EHIP, "result copy failed");
    return DTR_OK;
}

int dtr_sim_progress(dtr_sim *h, int64_t *ops_done)
{
    g_err.clear();
    if (!h || !ops_done) return fail(DTR_EINVAL, "null handle or output");
    *ops_done = 0;
    if (h->log || !h->last_queue) return DTR_OK;
    if (!h->progress_stream && hipStreamCreateWithFlags(&h->progress_stream, hipStreamNonBlocking) != hipSuccess) {
        h->progress_stream = nullptr;
        return fail(DTR_EHIP, "stream creation failed");
    }
    unsigned long long v = 0;
    if (hipMemcpyAsync(&v, (uint8_t *)h->last_queue + dtr::PROGRESS_OFFSET, sizeof v, hipMemcpyDeviceToHost,
                       h->progress_stream) != hipSuccess ||
        hipStreamSynchronize(h->progress_stream) != hipSuccess)
        return fail(DTR_EHIP, "progress read failed");
    *ops_done = (int64_t)v;
    return DTR_OK;
}

void dtr_sim_destroy(dtr_sim *h) { delete h; }

int dtr_log_workspace_bytes(const dtr_log *logs, int32_t n_logs, const dtr_sim_spec *sims, int32_t n_sims,
                            const dtr_sim_options *options, size_t *bytes)
{
    g_err.clear();
    if (!bytes) return fail(DTR_EINVAL, "null bytes");
    dtrhost::LogPlan *p = nullptr;
    if (int rc = dtrhost::log_plan_make(logs, n_logs, sims, n_sims, options, &p)) return rc;
    *bytes = dtrhost::log_plan_total(p);
    dtrhost::log_plan_free(p);
    return DTR_OK;
}

int dtr_log_create(const dtr_log *logs, int32_t n_logs, const dtr_sim_spec *sims, int32_t n_sims,
                   const dtr_sim_options *options, void *device_workspace, size_t workspace_bytes, void *stream,
                   dtr_sim **out)
{
    g_err.clear();
    if (!out) return fail(DTR_EINVAL, "null out");
    *out = nullptr;
    if (!device_workspace) return fail(DTR_EINVAL, "null device workspace");
    if ((uintptr_t)device_workspace % ALIGN) return fail(DTR_EINVAL, "workspace must be 256-byte aligned");
    dtr_sim *h = new dtr_sim();
    int rc = dtrhost::log_plan_make(logs, n_logs, sims, n_sims, options, &h->log);
    if (rc) { delete h; return rc; }
    const size_t need = dtrhost::log_plan_total(h->log);
    if (workspace_bytes < need) {
        rc = fail(DTR_EINVAL, "workspace too small: %zu bytes given, %zu needed", workspace_bytes, need);
        delete h;
        return rc;
    }
    h->ws = (uint8_t *)device_workspace;
    h->ws_bytes = workspace_bytes;
    h->n_sims = n_sims;
    rc = dtrhost::log_plan_upload(h->log, h->ws, (hipStream_t)stream);
    if (rc) { delete h; return rc; }
    *out = h;
    return DTR_OK;
}

int dtr_sim_launch_info(const dtr_sim *h, dtr_launch_info *out)
{
    g_err.clear();
    if (!h || !out) return fail(DTR_EINVAL, "null handle or output");
    out->reserved = 0;
    if (h->log) {
        dtrhost::log_plan_info(h->log, &out->n_slots, &out->waves_per_group, &out->lds_bytes);
    } else {
        out->n_slots = h->plan.n_slots;
        out->waves_per_group = h->plan.class_count[1] + h->plan.class_count[4] > 0 ? (int32_t)h->plan.L.walk_waves
                               : h->plan.class_count[0] > 0                      ? dtr::EQ_WAVES
                                                                                 : 1;
        if (h->plan.static_only)
            out->n_slots = (int32_t)std::max<int64_t>(1, std::min<int64_t>(
                out->n_slots, (int64_t)((DTR_STATIC_SCRATCH_BYTES - STATIC_HEADER) / (size_t)h->plan.L.bytes)));
        out->lds_bytes = 0;
    }
    return DTR_OK;
}

#ifdef DTR_PROFILE
// Phase timers of the last run (DTR_PROFILE builds only; not part of the
// public header): PROF_FIELDS int64 per simulation.
int dtr_sim_profile(dtr_sim *h, int64_t *host_out, int32_t n_sims)
{
    if (!h || h->log || n_sims != h->n_sims || !h->ran) return fail(DTR_EINVAL, "bad profile request");
    if (hipMemcpyAsync(host_out, h->ws + h->plan.prof_off, sizeof(int64_t) * dtr::PROF_FIELDS * n_sims,
                       hipMemcpyDeviceToHost, h->last_stream) != hipSuccess ||
        hipStreamSynchronize(h->last_stream) != hipSuccess)
        return fail(DTR_EHIP, "profile copy failed");
    return DTR_OK;
}
#endif

}  // extern "C"
