// dtr_log.cpp -- host side of operator-log replay (Appendix C.6): validation
// and lowering of DTR_LOG_* instruction streams to storages, tensors and
// operators (Appendix C.1), the per-storage metadata of Appendix C.2, the
// workspace plan, upload and launch.
//
// Lowering rules (the instruction semantics are stated in dtr_sim.h):
//   * every CALL, MUTATE and CONSTANT becomes one operator, numbered in log
//     order; CALL outputs are tensors that own a new storage or view one
//     (size 0); MUTATE outputs are clones that own new storages of the mutated
//     tensors' storage sizes, and the mutated names are rebound to them;
//     CONSTANT is an operator of cost 0 without inputs whose storage is
//     pinned from creation;
//   * names hold external references; COPY adds one, COPYFROM moves one,
//     RELEASE drops one; a storage whose last reference goes is released
//     after the latest operator (release events keep log order); tensors
//     still referenced at the end are required;
//   * a storage's cost c0 sums the cost of the operator of every tensor
//     viewing it, its parents are the storages those operators read (never
//     itself), its children are the reverse, all over the tensors that exist:
//     the first run of an operator creates its tensors, so the replay grows
//     costs and edges as it goes (the lists below are ordered for that); a
//     storage's dependents for banishing are the tensors (outside it)
//     computed by operators reading it.  Constant storages cost 0.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <unordered_set>
#include <vector>

#include "host.h"
#include "layout_log.h"

extern "C" hipError_t dtr_launch_log(const dtr::LogKernelArgs *args, hipStream_t stream);

namespace dtrhost {

namespace {

constexpr int64_t MAX_ITEMS = int64_t(1) << 26;    // storages, tensors, operators, list entries
constexpr int64_t MAX_C0_SUM = int64_t(1) << 50;    // keeps every score numerator below 2^51
constexpr size_t LDS_LIMIT = 160 * 1024;            // dynamic LDS of the log kernel (and the device's)

struct Lowered {
    int32_t S = 0, T = 0, F = 0;
    // storages
    std::vector<int64_t> s_size, s_c0;
    std::vector<uint8_t> s_const;
    std::vector<int32_t> par_off, par, ch_off, ch, dt_off, dt;
    std::vector<int32_t> born_off, born;   // per operator: edges its first run creates (parent, storage)
    // tensors
    std::vector<int32_t> t_storage, t_op;
    std::vector<uint8_t> t_alias;
    // operators
    std::vector<int64_t> op_cost, op_need;
    std::vector<int32_t> in_off{0}, in, ls_off, ls, out_off{0}, out, rel_off, rel;
    std::vector<int32_t> req;
};

class Lowerer {
public:
    Lowerer(const dtr_log &g, int32_t index, Lowered &L) : g_(g), idx_(index), L_(L) {}

    int run()
    {
        if (g_.n_instrs < 0 || g_.n_names < 0) return bad(-1, "negative n_instrs or n_names");
        if (g_.n_instrs > 0 && (!g_.kind || !g_.a || !g_.b || !g_.n_in || !g_.value || !g_.list_offsets))
            return fail(DTR_EINVAL, "log %d: null array", idx_);
        if (g_.n_instrs > 0 && g_.list_offsets[g_.n_instrs] > 0 && !g_.ids)
            return fail(DTR_EINVAL, "log %d: null ids", idx_);
        bound_.assign(g_.n_names, -1);
        out_mark_.assign(g_.n_names, -1);
        for (int32_t i = 0; i < g_.n_instrs;) {
            int rc = DTR_OK, step = 1;
            switch (g_.kind[i]) {
            case DTR_LOG_CONSTANT: rc = constant(i), step = 2; break;
            case DTR_LOG_CALL: rc = call(i, &step); break;
            case DTR_LOG_MUTATE: rc = mutate(i); break;
            case DTR_LOG_COPY: rc = copy(i); break;
            case DTR_LOG_COPYFROM: rc = copyfrom(i); break;
            case DTR_LOG_RELEASE: rc = release(i); break;
            default: return bad(i, "unexpected instruction kind %d", g_.kind[i]);
            }
            if (rc) return rc;
            i += step;
        }
        for (int32_t t = 0; t < (int32_t)t_ref_.size(); t++)
            if (t_ref_[t] > 0) L_.req.push_back(t);
        return derive();
    }

private:
    const dtr_log &g_;
    const int32_t idx_;
    Lowered &L_;
    std::vector<int32_t> bound_;       // name -> tensor, -1 unbound
    std::vector<int32_t> out_mark_;    // name -> operator that listed it as an output
    std::vector<int64_t> t_ref_, s_ref_;
    std::vector<int32_t> rel_op_;      // operator each release event follows

    __attribute__((format(printf, 3, 4))) int bad(int32_t i, const char *fmt, ...)
    {
        char msg[256];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(msg, sizeof(msg), fmt, ap);
        va_end(ap);
        if (i < 0) return fail(DTR_ETRACE, "log %d: %s", idx_, msg);
        return fail(DTR_ETRACE, "log %d, instruction %d: %s", idx_, i, msg);
    }
    bool name_ok(int32_t n) const { return n >= 0 && n < g_.n_names; }
    bool is_bound(int32_t n) const { return name_ok(n) && bound_[n] >= 0; }
    int32_t n_ops() const { return (int32_t)L_.op_cost.size(); }

    int32_t new_storage(int64_t size, bool constant)
    {
        L_.s_size.push_back(size);
        L_.s_const.push_back(constant ? 1 : 0);
        s_ref_.push_back(0);
        return (int32_t)L_.s_size.size() - 1;
    }
    int32_t new_tensor(int32_t storage, int32_t op, bool alias)
    {
        L_.t_storage.push_back(storage);
        L_.t_op.push_back(op);
        L_.t_alias.push_back(alias ? 1 : 0);
        t_ref_.push_back(0);
        return (int32_t)L_.t_storage.size() - 1;
    }
    // an operator's inputs and outputs are appended between begin_op and end_op
    int32_t begin_op(int64_t cost)
    {
        L_.op_cost.push_back(cost);
        return n_ops() - 1;
    }
    void end_op()
    {
        L_.in_off.push_back((int32_t)L_.in.size());
        L_.out_off.push_back((int32_t)L_.out.size());
    }
    void ref(int32_t t, int d)
    {
        t_ref_[t] += d;
        const int32_t s = L_.t_storage[t];
        s_ref_[s] += d;
        if (d < 0 && s_ref_[s] == 0) {     // every reference follows some operator
            L_.rel.push_back(s);
            rel_op_.push_back(n_ops() - 1);
        }
    }
    bool over_limit(int64_t more_inputs, int64_t more_outputs) const
    {
        return (int64_t)L_.s_size.size() + more_outputs >= MAX_ITEMS ||
               (int64_t)L_.t_storage.size() + more_outputs >= MAX_ITEMS || n_ops() + 1 >= MAX_ITEMS ||
               (int64_t)L_.in.size() + more_inputs >= MAX_ITEMS || (int64_t)L_.out.size() + more_outputs >= MAX_ITEMS;
    }
    int too_many(int32_t i) { return bad(i, "log exceeds 2^26 storages, tensors, operators or list entries"); }

    int constant(int32_t i)
    {
        const int32_t nm = g_.a[i];
        if (!name_ok(nm) || bound_[nm] >= 0) return bad(i, "constant name %d is not fresh", nm);
        if (i + 1 >= g_.n_instrs || g_.kind[i + 1] != DTR_LOG_MEMORY || g_.a[i + 1] != nm)
            return bad(i, "constant %d is not followed by its MEMORY", nm);
        const int64_t size = g_.value[i + 1];
        if (size < 1 || size >= MAX_SIZE) return bad(i + 1, "size %lld outside [1, 2^36)", (long long)size);
        if (over_limit(0, 1)) return too_many(i);
        const int32_t o = begin_op(0);
        const int32_t t = new_tensor(new_storage(size, true), o, false);
        L_.out.push_back(t);
        end_op();
        bound_[nm] = t;
        ref(t, +1);
        return DTR_OK;
    }

    int id_list(int32_t i, int64_t *lo, int32_t *nin, int64_t *nout)
    {
        *lo = g_.list_offsets[i];
        const int64_t hi = g_.list_offsets[i + 1];
        *nin = g_.n_in[i];
        if (*lo < 0 || hi < *lo || *nin < 0 || hi - *lo < *nin) return bad(i, "bad id list");
        *nout = hi - *lo - *nin;
        const int64_t cost = g_.value[i];
        if (cost < 1 || cost > MAX_COST) return bad(i, "cost %lld outside [1, 2^28]", (long long)cost);
        for (int64_t e = *lo; e < *lo + *nin; e++)
            if (!is_bound(g_.ids[e])) return bad(i, "input name %d is not bound", g_.ids[e]);
        if (over_limit(*nin, *nout)) return too_many(i);
        return DTR_OK;
    }

    int call(int32_t i, int *step)
    {
        int64_t lo, nout;
        int32_t nin;
        if (int rc = id_list(i, &lo, &nin, &nout)) return rc;
        if (nout < 1) return bad(i, "a call has no output");
        if ((int64_t)i + 2 * nout >= g_.n_instrs) return bad(i, "outputs are not all described");
        const int32_t o = begin_op(g_.value[i]);
        for (int64_t e = lo; e < lo + nin; e++) L_.in.push_back(bound_[g_.ids[e]]);
        // fresh-storage outputs of this call, by name (views may view them)
        std::vector<std::pair<int32_t, int32_t>> own;
        for (int64_t j = 0; j < nout; j++) {
            const int32_t nm = g_.ids[lo + nin + j];
            const int32_t mi = i + 1 + 2 * (int32_t)j, ai = mi + 1;
            if (!name_ok(nm) || bound_[nm] >= 0 || out_mark_[nm] == o)
                return bad(i, "output name %d is not fresh", nm);
            out_mark_[nm] = o;
            if (g_.kind[mi] != DTR_LOG_MEMORY || g_.a[mi] != nm || g_.kind[ai] != DTR_LOG_ALIAS || g_.a[ai] != nm)
                return bad(mi, "output %d is not described by MEMORY then ALIAS", nm);
            const int32_t src = g_.b[ai];
            int32_t t;
            if (src < 0) {
                const int64_t size = g_.value[mi];
                if (size < 1 || size >= MAX_SIZE) return bad(mi, "size %lld outside [1, 2^36)", (long long)size);
                t = new_tensor(new_storage(size, false), o, false);
                own.push_back({nm, t});
            } else {
                int32_t base = -1;
                for (auto &p : own)
                    if (p.first == src) base = p.second;
                if (base < 0 && is_bound(src))
                    for (int64_t e = lo; e < lo + nin; e++)
                        if (g_.ids[e] == src) base = bound_[src];
                if (base < 0) return bad(ai, "view of %d, which is neither an input nor a new output", src);
                t = new_tensor(L_.t_storage[base], o, true);
            }
            L_.out.push_back(t);
        }
        end_op();
        for (int64_t j = 0; j < nout; j++) {
            const int32_t nm = g_.ids[lo + nin + j];
            bound_[nm] = L_.out[L_.out.size() - nout + j];
            ref(bound_[nm], +1);
        }
        *step = 1 + 2 * (int)nout;
        return DTR_OK;
    }

    int mutate(int32_t i)
    {
        int64_t lo, nout;
        int32_t nin;
        if (int rc = id_list(i, &lo, &nin, &nout)) return rc;
        for (int64_t j = 0; j < nout; j++) {
            const int32_t nm = g_.ids[lo + nin + j];
            bool among = false, repeated = false;
            for (int64_t e = lo; e < lo + nin; e++) among |= g_.ids[e] == nm;
            for (int64_t q = lo + nin; q < lo + nin + j; q++) repeated |= g_.ids[q] == nm;
            if (!among || repeated) return bad(i, "mutated name %d is not a distinct input", nm);
        }
        const int32_t o = begin_op(g_.value[i]);
        for (int64_t e = lo; e < lo + nin; e++) L_.in.push_back(bound_[g_.ids[e]]);
        const size_t first = L_.out.size();
        for (int64_t j = 0; j < nout; j++) {
            const int32_t old = bound_[g_.ids[lo + nin + j]];
            L_.out.push_back(new_tensor(new_storage(L_.s_size[L_.t_storage[old]], false), o, false));
        }
        end_op();
        for (int64_t j = 0; j < nout; j++) {
            const int32_t nm = g_.ids[lo + nin + j];
            const int32_t old = bound_[nm];
            bound_[nm] = L_.out[first + j];
            ref(bound_[nm], +1);
            ref(old, -1);
        }
        return DTR_OK;
    }

    int copy(int32_t i)
    {
        const int32_t to = g_.a[i], from = g_.b[i];
        if (!name_ok(to) || bound_[to] >= 0 || !is_bound(from)) return bad(i, "copy %d <- %d", to, from);
        bound_[to] = bound_[from];
        ref(bound_[to], +1);
        return DTR_OK;
    }

    int copyfrom(int32_t i)
    {
        const int32_t to = g_.a[i], from = g_.b[i];
        if (!is_bound(to) || !is_bound(from)) return bad(i, "copyfrom %d <- %d", to, from);
        const int32_t old = bound_[to];
        bound_[to] = bound_[from];
        ref(bound_[to], +1);
        ref(old, -1);
        return DTR_OK;
    }

    int release(int32_t i)
    {
        const int32_t nm = g_.a[i];
        if (!is_bound(nm)) return bad(i, "release of unbound name %d", nm);
        const int32_t old = bound_[nm];
        bound_[nm] = -1;
        ref(old, -1);
        return DTR_OK;
    }

    static void csr(int32_t n, const std::vector<int32_t> &key, const std::vector<int32_t> &val,
                    std::vector<int32_t> &off, std::vector<int32_t> &out)
    {
        off.assign(n + 1, 0);
        for (int32_t k : key) off[k + 1]++;
        for (int32_t i = 0; i < n; i++) off[i + 1] += off[i];
        out.resize(val.size());
        std::vector<int32_t> fill(off.begin(), off.end() - 1);
        for (size_t z = 0; z < key.size(); z++) out[fill[key[z]]++] = val[z];
    }

    // per-operator and per-storage tables of the lowered program
    int derive()
    {
        Lowered &L = L_;
        const int32_t S = (int32_t)L.s_size.size(), T = (int32_t)L.t_storage.size(), F = n_ops();
        L.S = S;
        L.T = T;
        L.F = F;
        // release events: already grouped by operator, in log order
        L.rel_off.assign(F + 1, 0);
        for (int32_t o : rel_op_) L.rel_off[o + 1]++;
        for (int32_t o = 0; o < F; o++) L.rel_off[o + 1] += L.rel_off[o];
        // per operator: memory of its own new storages, distinct input storages
        L.op_need.assign(F, 0);
        L.ls_off.assign(F + 1, 0);
        std::vector<int32_t> seen(std::max(S, 1), -1);
        for (int32_t o = 0; o < F; o++) {
            for (int32_t q = L.out_off[o]; q < L.out_off[o + 1]; q++)
                if (!L.t_alias[L.out[q]]) L.op_need[o] += L.s_size[L.t_storage[L.out[q]]];
            for (int32_t e = L.in_off[o]; e < L.in_off[o + 1]; e++) {
                const int32_t s = L.t_storage[L.in[e]];
                if (seen[s] == o) continue;
                seen[s] = o;
                L.ls.push_back(s);
            }
            L.ls_off[o + 1] = (int32_t)L.ls.size();
        }
        // the storage graph in the order its edges appear: an operator's first
        // run creates its tensors, and each makes the storages the operator
        // reads parents of its own storage.  Both lists of every storage are
        // ordered by the operator creating the edge, so the edges that exist
        // at any time are a prefix; born_* lists each operator's new edges.
        // The costs of the storages at the end bound every score.
        L.s_c0.assign(S, 0);
        int64_t c0_sum = 0;
        for (int32_t t = 0; t < T; t++) {
            const int32_t st = L.t_storage[t];
            if (L.s_const[st]) continue;
            L.s_c0[st] += L.op_cost[L.t_op[t]];     // a term per tensor of the storage
            c0_sum += L.op_cost[L.t_op[t]];
            if (c0_sum >= MAX_C0_SUM) return bad(-1, "storage costs sum to 2^50 or more");
        }
        {
            std::unordered_set<uint64_t> edges;
            std::vector<int32_t> pk, pv, ck, cv;    // (storage, neighbour) in creation order
            L.born_off.assign(F + 1, 0);
            for (int32_t o = 0; o < F; o++) {
                for (int32_t q = L.out_off[o]; q < L.out_off[o + 1]; q++) {
                    const int32_t st = L.t_storage[L.out[q]];
                    for (int32_t e = L.ls_off[o]; e < L.ls_off[o + 1]; e++) {
                        const int32_t par = L.ls[e];
                        if (par == st || !edges.insert(((uint64_t)(uint32_t)par << 32) | (uint32_t)st).second)
                            continue;
                        pk.push_back(st);
                        pv.push_back(par);
                        ck.push_back(par);
                        cv.push_back(st);
                        L.born.push_back(par);
                        L.born.push_back(st);
                        if ((int64_t)pk.size() >= MAX_ITEMS) return bad(-1, "storage graph exceeds 2^26 edges");
                    }
                }
                L.born_off[o + 1] = (int32_t)(L.born.size() / 2);
            }
            csr(S, pk, pv, L.par_off, L.par);       // a stable fill keeps creation order
            csr(S, ck, cv, L.ch_off, L.ch);
        }
        // banishing dependents: outputs (outside p) of every operator reading p
        {
            std::vector<int32_t> key, val;
            for (int32_t o = 0; o < F; o++)
                for (int32_t e = L.ls_off[o]; e < L.ls_off[o + 1]; e++)
                    for (int32_t q = L.out_off[o]; q < L.out_off[o + 1]; q++)
                        if (L.t_storage[L.out[q]] != L.ls[e]) {
                            key.push_back(L.ls[e]);
                            val.push_back(L.out[q]);
                            if ((int64_t)key.size() >= MAX_ITEMS) return bad(-1, "dependent lists exceed 2^26");
                        }
            csr(S, key, val, L.dt_off, L.dt);
        }
        return DTR_OK;
    }
};

template <class T>
size_t bytes_of(const std::vector<T> &v) { return align_up(v.size() * sizeof(T)); }

size_t log_bytes(const Lowered &d)
{
    return bytes_of(d.s_size) + bytes_of(d.s_c0) + bytes_of(d.s_const) + bytes_of(d.par_off) + bytes_of(d.par) +
           bytes_of(d.ch_off) + bytes_of(d.ch) + bytes_of(d.dt_off) + bytes_of(d.dt) + bytes_of(d.t_storage) +
           bytes_of(d.t_op) + bytes_of(d.t_alias) + bytes_of(d.op_cost) + bytes_of(d.op_need) +
           bytes_of(d.in_off) + bytes_of(d.in) + bytes_of(d.ls_off) + bytes_of(d.ls) + bytes_of(d.out_off) +
           bytes_of(d.out) + bytes_of(d.rel_off) + bytes_of(d.rel) + bytes_of(d.req) + bytes_of(d.born_off) +
           bytes_of(d.born) + 26 * ALIGN;
}

}  // namespace

struct LogPlan {
    std::vector<Lowered> logs;
    std::vector<dtr_sim_spec> sims;
    std::vector<int32_t> order;
    dtr::LogSlotLayout L{};
    int32_t n_slots = 1;
    int32_t lds_bytes = 0, lds_state = 0, lds_wm = 0, lds_po = 0, lds_co = 0, lds_pa = 0, lds_ca = 0, wm_words = 0;
    int32_t lds_c0 = 0, lds_cand = 0, lds_stk = 0, lds_ctr = 0, lds_sz = 0, lds_last = 0, lds_rsum = 0, lds_rcnt = 0;
    int32_t lds_pcnt = 0, lds_ccnt = 0, lds_ctl = 0, waves = 1;
    std::vector<size_t> log_off;
    size_t desc_off = 0, spec_off = 0, order_off = 0, tables_bytes = 0, result_off = 0, slot_off = 0, total = 0;
};

int log_plan_make(const dtr_log *logs, int32_t n_logs, const dtr_sim_spec *sims, int32_t n_sims,
                  const dtr_sim_options *opt, LogPlan **out)
{
    *out = nullptr;
    if (n_logs < 0 || n_sims < 0) return fail(DTR_EINVAL, "negative n_logs or n_sims");
    if ((n_logs > 0 && !logs) || (n_sims > 0 && !sims)) return fail(DTR_EINVAL, "null logs or sims");
    if (opt && (opt->slots < 0 || (opt->flags & ~DTR_OPT_LOG_NO_LDS))) return fail(DTR_EINVAL, "bad options");
    LogPlan *p = new LogPlan();
    auto give_up = [&](int rc) { delete p; return rc; };
    p->logs.resize(n_logs);
    for (int32_t i = 0; i < n_logs; i++) {
        Lowerer lw(logs[i], i, p->logs[i]);
        if (int rc = lw.run()) return give_up(rc);
    }
    bool need_uf = false, need_walk = false;
    int64_t S_max = 1, T_max = 1, F_max = 1, E_max = 0;
    for (int32_t i = 0; i < n_sims; i++) {
        const dtr_sim_spec &s = sims[i];
        if (s.trace < 0 || s.trace >= n_logs) return give_up(fail(DTR_ETRACE, "sim %d: log index %d out of range", i, s.trace));
        if (int rc = check_spec(s, i)) return give_up(rc);
        need_uf |= heuristic_class(s.heuristic) == 0;
        need_walk |= heuristic_class(s.heuristic) == 1;
        const Lowered &d = p->logs[s.trace];
        S_max = std::max<int64_t>(S_max, d.S);
        T_max = std::max<int64_t>(T_max, d.T);
        F_max = std::max<int64_t>(F_max, d.F);
        E_max = std::max<int64_t>(E_max, (int64_t)d.par.size());
    }
    p->sims.assign(sims, sims + n_sims);
    // walk state in LDS when the largest log fits: storage states, visited
    // bitsets, storage graph with 16-bit neighbour ids.  With walk heuristics
    // the workgroup takes up to MAX_LOG_WAVES waves (helpers in the walk
    // scans), each with its own bitsets and stacks, as many as fit.
    const int64_t W = (S_max + 127) / 128 * 4;     // 32-bit words, whole 16-byte quads
    {
        int dev = 0, lds_max = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
            return give_up(fail(DTR_EHIP, "hipDeviceGetAttribute(maxSharedMemoryPerBlock) failed"));
        const size_t limit = std::min<size_t>(LDS_LIMIT, (size_t)lds_max);
        p->lds_bytes = 0;
        p->waves = 1;
        for (int32_t nw = need_walk ? dtr::MAX_LOG_WAVES : 1; nw >= 1; nw /= 2) {
            const size_t lanes = (size_t)dtr::WAVE * (size_t)nw;
            size_t q = 0;
            auto at = [&](int32_t &field, size_t bytes) { field = (int32_t)q; q += (bytes + 15) / 16 * 16; };
            at(p->lds_state, (size_t)S_max);
            at(p->lds_wm, 4 * (size_t)W * lanes);
            at(p->lds_po, 4 * (size_t)(S_max + 1));
            at(p->lds_co, 4 * (size_t)(S_max + 1));
            at(p->lds_pa, 2 * (size_t)E_max);
            at(p->lds_ca, 2 * (size_t)E_max);
            at(p->lds_c0, 8 * (size_t)S_max);
            at(p->lds_cand, 2 * (size_t)S_max);
            at(p->lds_stk, 2 * (size_t)dtr::LOG_LDS_STACK * lanes);
            at(p->lds_ctr, 4);
            at(p->lds_ctl, 16);
            at(p->lds_sz, 8 * (size_t)S_max);
            at(p->lds_last, 8 * (size_t)S_max);
            at(p->lds_rsum, 8 * (size_t)S_max);
            at(p->lds_rcnt, 4 * (size_t)S_max);
            at(p->lds_pcnt, 4 * (size_t)S_max);
            at(p->lds_ccnt, 4 * (size_t)S_max);
            const bool fits = S_max <= 65535 && q <= limit && !(opt && (opt->flags & DTR_OPT_LOG_NO_LDS));
            if (fits) {
                p->lds_bytes = (int32_t)q;
                p->waves = nw;
                break;
            }
        }
        p->wm_words = (int32_t)W;
    }
    // slot layout
    dtr::LogSlotLayout &L = p->L;
    size_t o = 0;
    auto take = [&](int64_t &field, size_t bytes) { field = (int64_t)o; o += align_up(bytes); };
    L.S_max = S_max;
    L.T_max = T_max;
    L.F_max = F_max;
    L.ucap = need_uf ? 2 * S_max + 64 : 0;
    L.mcap = L.ucap;
    const size_t S = (size_t)S_max, U = (size_t)L.ucap;
    take(L.state, S);
    take(L.pinned, S);
    take(L.pending, S);
    take(L.locks, 4 * S);
    take(L.node, 4 * S);
    take(L.sgen, 8 * S);
    take(L.last, 8 * S);
    take(L.gen, 8 * (size_t)T_max);
    take(L.c0d, 8 * S);
    take(L.pcnt, 4 * S);
    take(L.ccnt, 4 * S);
    take(L.uf_parent, 4 * U);
    take(L.uf_size, 4 * U);
    take(L.uf_remap, 4 * U);
    take(L.uf_cost, 8 * U);
    take(L.uf_tmp, 8 * U);
    take(L.mark, 4 * (size_t)L.mcap * dtr::WAVE);
    take(L.wmark, need_walk ? 4 * (size_t)W * dtr::WAVE : 0);
    take(L.queue, need_walk ? 4 * (S + 2) * dtr::WAVE * (size_t)p->waves : 0);     // per lane of every wave
    take(L.stack, sizeof(dtr::LogFrame) * (size_t)(F_max + 2));
    L.bytes = (int64_t)o;

    int32_t cus = 0;
    if (int rc = device_cus(&cus)) return give_up(rc);
    int64_t slots = opt && opt->slots > 0 ? opt->slots : (int64_t)cus * 16;
    const int64_t cap_bytes = int64_t(48) << 30;     // bound slot memory
    slots = std::min<int64_t>(slots, std::max<int64_t>(1, cap_bytes / std::max<int64_t>(1, L.bytes)));
    slots = std::min<int64_t>(slots, std::max<int32_t>(1, n_sims));
    p->n_slots = (int32_t)std::max<int64_t>(1, slots);

    // longest logs first, then lower budget first
    p->order.resize(n_sims);
    std::iota(p->order.begin(), p->order.end(), 0);
    std::stable_sort(p->order.begin(), p->order.end(), [&](int32_t a, int32_t b) {
        const int32_t fa = p->logs[sims[a].trace].F, fb = p->logs[sims[b].trace].F;
        if (fa != fb) return fa > fb;
        return sims[a].budget < sims[b].budget;
    });

    size_t w = align_up(64);   // header: work counter
    p->log_off.resize(n_logs);
    for (int32_t i = 0; i < n_logs; i++) {
        p->log_off[i] = w;
        w += log_bytes(p->logs[i]);
    }
    p->desc_off = w;
    w += align_up(sizeof(dtr::LogProgDev) * std::max(1, n_logs));
    p->spec_off = w;
    w += align_up(sizeof(dtr::SpecDev) * std::max(1, n_sims));
    p->order_off = w;
    w += align_up(sizeof(int32_t) * std::max(1, n_sims));
    p->tables_bytes = w;
    p->result_off = w;
    w += align_up(sizeof(dtr::ResultDev) * std::max(1, n_sims));
    p->slot_off = w;
    w += (size_t)L.bytes * (size_t)p->n_slots;
    p->total = w;
    *out = p;
    return DTR_OK;
}

size_t log_plan_total(const LogPlan *p) { return p->total; }
void log_plan_info(const LogPlan *p, int32_t *n_slots, int32_t *waves, int32_t *lds_bytes)
{
    *n_slots = p->n_slots;
    *waves = p->lds_bytes > 0 ? p->waves : 1;
    *lds_bytes = p->lds_bytes;
}
size_t log_plan_result_off(const LogPlan *p) { return p->result_off; }
void log_plan_free(LogPlan *p) { delete p; }

int log_plan_upload(LogPlan *p, uint8_t *ws, hipStream_t st)
{
    std::vector<uint8_t> staging(p->tables_bytes, 0);
    uint8_t *H = staging.data();
    const int32_t n_logs = (int32_t)p->logs.size(), n_sims = (int32_t)p->sims.size();
    std::vector<dtr::LogProgDev> descs(std::max(1, n_logs));
    for (int32_t i = 0; i < n_logs; i++) {
        const Lowered &d = p->logs[i];
        size_t w = p->log_off[i];
        auto put = [&](const auto &v) {
            using T = typename std::decay_t<decltype(v)>::value_type;
            const size_t at = w;
            if (!v.empty()) std::memcpy(H + at, v.data(), v.size() * sizeof(T));
            w += bytes_of(v);
            return (const T *)(ws + at);
        };
        dtr::LogProgDev &D = descs[i];
        D.S = d.S;
        D.T = d.T;
        D.F = d.F;
        D.n_req = (int32_t)d.req.size();
        D.s_size = put(d.s_size);
        D.s_c0 = put(d.s_c0);
        D.s_const = put(d.s_const);
        D.par_off = put(d.par_off);
        D.par = put(d.par);
        D.ch_off = put(d.ch_off);
        D.ch = put(d.ch);
        D.dt_off = put(d.dt_off);
        D.dt = put(d.dt);
        D.t_storage = put(d.t_storage);
        D.t_op = put(d.t_op);
        D.t_alias = put(d.t_alias);
        D.op_cost = put(d.op_cost);
        D.op_need = put(d.op_need);
        D.in_off = put(d.in_off);
        D.in = put(d.in);
        D.ls_off = put(d.ls_off);
        D.ls = put(d.ls);
        D.out_off = put(d.out_off);
        D.out = put(d.out);
        D.rel_off = put(d.rel_off);
        D.rel = put(d.rel);
        D.req = put(d.req);
        D.born_off = put(d.born_off);
        D.born = put(d.born);
    }
    std::memcpy(H + p->desc_off, descs.data(), sizeof(dtr::LogProgDev) * n_logs);
    for (int32_t i = 0; i < n_sims; i++) {
        const dtr_sim_spec &s = p->sims[i];
        dtr::SpecDev d{s.trace, s.heuristic, s.budget, s.seed, s.policy, s.search};
        std::memcpy(H + p->spec_off + i * sizeof(dtr::SpecDev), &d, sizeof(d));
    }
    if (n_sims) std::memcpy(H + p->order_off, p->order.data(), sizeof(int32_t) * n_sims);
    if (hipMemcpyAsync(ws, H, p->tables_bytes, hipMemcpyHostToDevice, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return fail(DTR_EHIP, "upload of %zu bytes failed", p->tables_bytes);
    return DTR_OK;
}

int log_plan_launch(const LogPlan *p, uint8_t *ws, hipStream_t st)
{
    dtr::LogKernelArgs a;
    a.progs = (const dtr::LogProgDev *)(ws + p->desc_off);
    a.specs = (const dtr::SpecDev *)(ws + p->spec_off);
    a.order = (const int32_t *)(ws + p->order_off);
    a.results = (dtr::ResultDev *)(ws + p->result_off);
    a.queue = (uint32_t *)ws;
    a.slots = ws + p->slot_off;
    a.L = p->L;
    a.n_sims = (int32_t)p->sims.size();
    a.n_slots = p->n_slots;
    a.lds_bytes = p->lds_bytes;
    a.lds_state = p->lds_state;
    a.lds_wm = p->lds_wm;
    a.lds_po = p->lds_po;
    a.lds_co = p->lds_co;
    a.lds_pa = p->lds_pa;
    a.lds_ca = p->lds_ca;
    a.wm_words = p->wm_words;
    a.lds_c0 = p->lds_c0;
    a.lds_cand = p->lds_cand;
    a.lds_stk = p->lds_stk;
    a.lds_ctr = p->lds_ctr;
    a.lds_sz = p->lds_sz;
    a.lds_last = p->lds_last;
    a.lds_rsum = p->lds_rsum;
    a.lds_rcnt = p->lds_rcnt;
    a.lds_pcnt = p->lds_pcnt;
    a.lds_ccnt = p->lds_ccnt;
    a.lds_ctl = p->lds_ctl;
    a.waves = p->waves;
    hipError_t e = dtr_launch_log(&a, st);
    if (e != hipSuccess) return fail(DTR_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
    return DTR_OK;
}

}  // namespace dtrhost
