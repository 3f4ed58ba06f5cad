/*
 * A plain C client of the library's host entry points (no GPU needed): the
 * bucket planner, its queries, the status strings and the auto-wrapping
 * planner.  Reads the buckets to plan from stdin and prints what the library
 * returns, one fact per line, for the test that runs it to compare with the
 * oracle.
 *
 * Input:   W P align  dim0_0 inner_0 ... dim0_{P-1} inner_{P-1}   (one plan per line)
 *          then a line "wrap n backward alpha_ag beta_ag alpha_rs beta_rs mem_max"
 *          followed by n lines "ag_words rs_words compute_time compute_mem".
 * Output:  plan <status> S=<S>
 *          param <p> c=<c_p> off=<off_p> L=<L_p> rows=<n_{p,0}>,...,<n_{p,W-1}>
 *          wrap <status> buckets=<k> of=<b_0>,...,<b_{n-1}>
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "fsdp_bucket.h"

static int plan_line(const char* line) {
    int W, P, A, used = 0, off = 0;
    if (sscanf(line, "%d %d %d%n", &W, &P, &A, &used) != 3) return -1;
    off += used;
    int64_t* dim0 = calloc(P > 0 ? P : 1, sizeof(int64_t));
    int64_t* inner = calloc(P > 0 ? P : 1, sizeof(int64_t));
    for (int p = 0; p < P; ++p) {
        long long n, k;
        if (sscanf(line + off, "%lld %lld%n", &n, &k, &used) != 2) { free(dim0); free(inner); return -1; }
        off += used;
        dim0[p] = n;
        inner[p] = k;
    }
    fsdp_plan* plan = NULL;
    fsdp_status st = fsdp_bucket_plan(W, P, dim0, inner, A, &plan);
    printf("plan %d S=%lld\n", (int)st, st == FSDP_OK ? (long long)fsdp_plan_chunk_elems(plan) : -1LL);
    if (st != FSDP_OK) {
        printf("error %s | %s\n", fsdp_status_str(st), fsdp_last_error());
    } else {
        for (int p = 0; p < P; ++p) {
            int64_t c, o, L;
            fsdp_plan_param(plan, p, &c, &o, &L);
            printf("param %d c=%lld off=%lld L=%lld rows=", p, (long long)c, (long long)o, (long long)L);
            for (int r = 0; r < W; ++r)
                printf("%s%lld", r ? "," : "", (long long)fsdp_plan_local_rows(plan, p, r));
            printf("\n");
        }
        fsdp_plan_free(plan);
    }
    free(dim0);
    free(inner);
    return 0;
}

static int wrap_block(const char* head, FILE* in) {
    int n, backward;
    double a_ag, b_ag, a_rs, b_rs;
    long long mem_max;
    if (sscanf(head, "wrap %d %d %lf %lf %lf %lf %lld", &n, &backward, &a_ag, &b_ag, &a_rs, &b_rs, &mem_max) != 7)
        return -1;
    const int m = n > 0 ? n : 1;
    int64_t* ag = calloc(m, sizeof(int64_t));
    int64_t* rs = calloc(m, sizeof(int64_t));
    double* t = calloc(m, sizeof(double));
    int64_t* mem = calloc(m, sizeof(int64_t));
    int32_t* of = calloc(m, sizeof(int32_t));
    for (int i = 0; i < n; ++i) {
        long long x, y, z;
        if (fscanf(in, "%lld %lld %lf %lld", &x, &y, &t[i], &z) != 4) return -1;
        ag[i] = x;
        rs[i] = y;
        mem[i] = z;
    }
    int32_t nb = -1;
    fsdp_status st = fsdp_auto_wrap(n, backward, ag, rs, t, mem, a_ag, b_ag, a_rs, b_rs, mem_max, of, &nb);
    printf("wrap %d buckets=%d of=", (int)st, (int)nb);
    for (int i = 0; st == FSDP_OK && i < n; ++i) printf("%s%d", i ? "," : "", (int)of[i]);
    printf("\n");
    free(ag); free(rs); free(t); free(mem); free(of);
    return 0;
}

int main(void) {
    char line[1 << 16];
    while (fgets(line, sizeof line, stdin)) {
        if (strncmp(line, "wrap", 4) == 0) {
            if (wrap_block(line, stdin) != 0) return 2;
        } else if (line[0] != '\n' && plan_line(line) != 0) {
            return 2;
        }
    }
    return 0;
}
