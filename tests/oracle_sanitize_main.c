/*
 * oracle_sanitize_main.c -- a stand-alone driver of the CPU oracle, built by
 * tests/test_sanitize.py with AddressSanitizer and UndefinedBehaviorSanitizer
 * (a sanitized shared library loaded into Python would miss the interposed
 * allocator).  Test infrastructure only: it includes the oracle's source.
 *
 * Input file (little-endian): the traces, their simulations, the operator
 * logs and their simulations, each array in full:
 *   int32 n_traces; per trace: int32 n_tensors, n_ops; int64 size[n];
 *     uint8 flags[n]; int32 out[F]; int64 cost[F]; int64 off[F+1];
 *     int32 in[off[F]]
 *   int32 n_sims; oracle_spec[n_sims] (32 bytes each)
 *   int32 n_logs; per log: int32 n_instrs, n_names; int32 kind[m], a[m],
 *     b[m], n_in[m]; int64 value[m]; int64 list_offsets[m+1];
 *     int32 ids[list_offsets[m]]
 *   int32 n_log_sims; oracle_spec[n_log_sims]
 * Output file: the trace results, then the log results (R_NFIELDS int64 each).
 * Usage: oracle_sanitize_main <in> <out> <threads>
 */
#include "../oracle/dtr_oracle.c"

#include <stdio.h>

static FILE *in_f;

static void *read_n(size_t bytes)
{
    void *p = malloc(bytes ? bytes : 1);
    if (!p || (bytes && fread(p, 1, bytes, in_f) != bytes)) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return p;
}

static int32_t read_i32(void)
{
    int32_t *p = read_n(4);
    int32_t v = *p;
    free(p);
    return v;
}

int main(int argc, char **argv)
{
    if (argc != 4) return 2;
    in_f = fopen(argv[1], "rb");
    if (!in_f) return 2;
    int32_t threads = (int32_t)atoi(argv[3]);

    int32_t nt = read_i32();
    oracle_trace *tr = calloc((size_t)(nt > 0 ? nt : 1), sizeof(oracle_trace));
    for (int32_t i = 0; i < nt; i++) {
        tr[i].n_tensors = read_i32();
        tr[i].n_ops = read_i32();
        size_t n = (size_t)tr[i].n_tensors, f = (size_t)tr[i].n_ops;
        tr[i].tensor_size = read_n(8 * n);
        tr[i].tensor_flags = read_n(n);
        tr[i].op_output = read_n(4 * f);
        tr[i].op_cost = read_n(8 * f);
        int64_t *off = read_n(8 * (f + 1));
        tr[i].op_input_offsets = off;
        tr[i].op_inputs = read_n(4 * (size_t)off[f]);
    }
    int32_t ns = read_i32();
    oracle_spec *sp = read_n(sizeof(oracle_spec) * (size_t)ns);
    int32_t nl = read_i32();
    oracle_log *lg = calloc((size_t)(nl > 0 ? nl : 1), sizeof(oracle_log));
    for (int32_t i = 0; i < nl; i++) {
        lg[i].n_instrs = read_i32();
        lg[i].n_names = read_i32();
        size_t m = (size_t)lg[i].n_instrs;
        lg[i].kind = read_n(4 * m);
        lg[i].a = read_n(4 * m);
        lg[i].b = read_n(4 * m);
        lg[i].n_in = read_n(4 * m);
        lg[i].value = read_n(8 * m);
        int64_t *lo = read_n(8 * (m + 1));
        lg[i].list_offsets = lo;
        lg[i].ids = read_n(4 * (size_t)lo[m]);
    }
    int32_t nls = read_i32();
    oracle_spec *lsp = read_n(sizeof(oracle_spec) * (size_t)nls);
    fclose(in_f);

    int64_t *res = calloc((size_t)(ns > 0 ? ns : 1) * R_NFIELDS, sizeof(int64_t));
    int64_t *lres = calloc((size_t)(nls > 0 ? nls : 1) * R_NFIELDS, sizeof(int64_t));
    int rc = oracle_run(tr, nt, sp, ns, res, threads, NULL);
    int rc2 = oracle_run_log(lg, nl, lsp, nls, lres, threads);
    if (rc || rc2) {
        fprintf(stderr, "oracle returned %d / %d\n", rc, rc2);
        return 3;
    }
    FILE *out = fopen(argv[2], "wb");
    if (!out) return 2;
    fwrite(res, sizeof(int64_t), (size_t)ns * R_NFIELDS, out);
    fwrite(lres, sizeof(int64_t), (size_t)nls * R_NFIELDS, out);
    fclose(out);

    for (int32_t i = 0; i < nt; i++) {
        free((void *)tr[i].tensor_size);
        free((void *)tr[i].tensor_flags);
        free((void *)tr[i].op_output);
        free((void *)tr[i].op_cost);
        free((void *)tr[i].op_input_offsets);
        free((void *)tr[i].op_inputs);
    }
    for (int32_t i = 0; i < nl; i++) {
        free((void *)lg[i].kind);
        free((void *)lg[i].a);
        free((void *)lg[i].b);
        free((void *)lg[i].n_in);
        free((void *)lg[i].value);
        free((void *)lg[i].list_offsets);
        free((void *)lg[i].ids);
    }
    free(tr);
    free(lg);
    free(sp);
    free(lsp);
    free(res);
    free(lres);
    return 0;
}
