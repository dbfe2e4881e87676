// host_sanitize_main.cpp -- a stand-alone driver of the library's host code
// (trace validation and derivation, operator-log validation and lowering,
// workspace layout), built by tests/test_sanitize.py with AddressSanitizer
// and UndefinedBehaviorSanitizer.  The device entry points of the kernel
// sources are replaced by stubs that report no device: sizing a workspace
// runs every host step, then stops with DTR_EHIP where a device is queried.
//
// Input file: as for oracle_sanitize_main.c.  Prints the return codes of
// dtr_sim_workspace_bytes (all traces, all their simulations) and of
// dtr_log_workspace_bytes (all logs, all their simulations).
// Usage: host_sanitize_main <in>
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "dtr_sim.h"

namespace dtr { struct KernelArgs; struct LogKernelArgs; }
extern "C" hipError_t dtr_launch_reset(uint32_t *, hipStream_t) { return hipErrorNoDevice; }
extern "C" hipError_t dtr_launch_group(const dtr::KernelArgs *, int32_t, hipStream_t) { return hipErrorNoDevice; }
extern "C" hipError_t dtr_launch_log(const dtr::LogKernelArgs *, hipStream_t) { return hipErrorNoDevice; }
extern "C" hipError_t dtr_static_scratch(void **, size_t *) { return hipErrorNoDevice; }

static FILE *in_f;
static std::vector<std::vector<char>> keep;

static const void *read_n(size_t bytes)
{
    keep.emplace_back(bytes ? bytes : 1);
    if (bytes && fread(keep.back().data(), 1, bytes, in_f) != bytes) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return keep.back().data();
}

static int32_t read_i32() { return *(const int32_t *)read_n(4); }

int main(int argc, char **argv)
{
    if (argc != 2) return 2;
    in_f = fopen(argv[1], "rb");
    if (!in_f) return 2;
    const int32_t nt = read_i32();
    std::vector<dtr_trace> tr(nt > 0 ? nt : 1);
    for (int32_t i = 0; i < nt; i++) {
        tr[i].n_tensors = read_i32();
        tr[i].n_ops = read_i32();
        const size_t n = (size_t)tr[i].n_tensors, f = (size_t)tr[i].n_ops;
        tr[i].tensor_size = (const int64_t *)read_n(8 * n);
        tr[i].tensor_flags = (const uint8_t *)read_n(n);
        tr[i].op_output = (const int32_t *)read_n(4 * f);
        tr[i].op_cost = (const int64_t *)read_n(8 * f);
        tr[i].op_input_offsets = (const int64_t *)read_n(8 * (f + 1));
        tr[i].op_inputs = (const int32_t *)read_n(4 * (size_t)tr[i].op_input_offsets[f]);
    }
    const int32_t ns = read_i32();
    const dtr_sim_spec *sp = (const dtr_sim_spec *)read_n(sizeof(dtr_sim_spec) * (size_t)ns);
    const int32_t nl = read_i32();
    std::vector<dtr_log> lg(nl > 0 ? nl : 1);
    for (int32_t i = 0; i < nl; i++) {
        lg[i].n_instrs = read_i32();
        lg[i].n_names = read_i32();
        const size_t m = (size_t)lg[i].n_instrs;
        lg[i].kind = (const int32_t *)read_n(4 * m);
        lg[i].a = (const int32_t *)read_n(4 * m);
        lg[i].b = (const int32_t *)read_n(4 * m);
        lg[i].n_in = (const int32_t *)read_n(4 * m);
        lg[i].value = (const int64_t *)read_n(8 * m);
        lg[i].list_offsets = (const int64_t *)read_n(8 * (m + 1));
        lg[i].ids = (const int32_t *)read_n(4 * (size_t)lg[i].list_offsets[m]);
    }
    const int32_t nls = read_i32();
    const dtr_sim_spec *lsp = (const dtr_sim_spec *)read_n(sizeof(dtr_sim_spec) * (size_t)nls);
    fclose(in_f);
    size_t bytes = 0;
    const int rc = dtr_sim_workspace_bytes(tr.data(), nt, sp, ns, nullptr, &bytes);
    printf("%d\n", rc);
    const int rc2 = dtr_log_workspace_bytes(lg.data(), nl, lsp, nls, nullptr, &bytes);
    printf("%d\n", rc2);
    return 0;
}
