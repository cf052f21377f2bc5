/*
 * A plain C99 client of rc_cohort.h on the GPU: device memory from
 * hipMalloc, no Python and no torch, exactly as a C caller would use the
 * library.  Inputs are drawn here from a SplitMix64 stream; the expected
 * outputs come from the oracle's C entry point (test infrastructure, linked
 * only by this test).  Each shape reaches one kernel form:
 *   - W = 32, 300 cohorts of 256, mod-256 routes: the two-role split;
 *   - W = 64, mixed cohorts of 32..256, 1024 CDF routes: the table image;
 *   - W = 16, one cohort of 64, mod-16 routes: the pipelined split;
 *   - W = 8, 32 cohorts of 32, mod-4 routes, one step: the one-lane chain.
 * For each: the resident chain over all cohorts and over three ragged cohort
 * ranges, the host round trip, and the allocation-free entry point in both
 * mechanisms, each compared with the oracle bit for bit (padding columns
 * included), plus the library's launch and copy counters.
 * Prints "ok" and exits 0 when every check holds; otherwise names the check
 * that failed and exits 1.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "rc_cohort.h"

/* the oracle's C entry point (oracle/rc_oracle.c) */
int rc_oracle_run_chain(uint32_t n_sessions, uint32_t n_words, uint32_t n_routes,
                        uint32_t n_cohorts, const uint32_t *cohort_offsets,
                        const uint32_t *table, uint32_t route_mode, const uint32_t *route_cdf,
                        uint32_t decide_thr, uint32_t *state, uint32_t *outcome,
                        uint32_t *eff_sid, uint32_t *eff_tool, uint32_t *eff_payload,
                        uint32_t *n_taken, uint32_t ld, uint32_t step0, uint32_t n_steps,
                        uint32_t cohort_begin, uint32_t cohort_end, uint32_t *decisions_out);

static int failures = 0;

static void check(int cond, const char *shape, const char *what) {
    if (!cond) {
        printf("FAILED: %s: %s\n", shape, what);
        fflush(stdout);
        ++failures;
    }
}

/* SplitMix64 (Steele, Lea and Flood, 2014); the high half of each output */
static uint64_t sm_state;
static uint32_t next_u32(void) {
    uint64_t z = (sm_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return (uint32_t)((z ^ (z >> 31)) >> 32);
}

typedef struct {
    const char *name;
    uint32_t W, R, route_mode, thr, T, step0;
    uint32_t n_cohorts;
    const uint32_t *size_cycle; /* cohort sizes, repeated */
    uint32_t n_cycle;
} Shape;

/* host copies of the six buffers */
typedef struct {
    uint32_t *state, *outcome, *sid, *tool, *pay, *cnt;
    size_t n_state, n_outcome, n_eff, n_pay, n_cnt;
} Host;

static int host_alloc(Host *h, uint32_t W, uint32_t ld, uint32_t T, uint32_t C) {
    h->n_state = (size_t)W * ld;
    h->n_outcome = ld;
    h->n_eff = (size_t)T * ld;
    h->n_pay = (size_t)T * ld * 4u;
    h->n_cnt = (size_t)T * C;
    h->state = malloc(h->n_state * 4u);
    h->outcome = malloc(h->n_outcome * 4u);
    h->sid = malloc(h->n_eff * 4u);
    h->tool = malloc(h->n_eff * 4u);
    h->pay = malloc(h->n_pay * 4u);
    h->cnt = malloc(h->n_cnt * 4u);
    return h->state && h->outcome && h->sid && h->tool && h->pay && h->cnt;
}

static void host_free(Host *h) {
    free(h->state);
    free(h->outcome);
    free(h->sid);
    free(h->tool);
    free(h->pay);
    free(h->cnt);
}

static void fill_outputs(Host *h) {
    memset(h->sid, 0xFF, h->n_eff * 4u);
    memset(h->tool, 0xFF, h->n_eff * 4u);
    memset(h->pay, 0xFF, h->n_pay * 4u);
    memset(h->cnt, 0xFF, h->n_cnt * 4u);
}

static int same(const Host *a, const Host *b) {
    return memcmp(a->state, b->state, a->n_state * 4u) == 0 &&
           memcmp(a->outcome, b->outcome, a->n_outcome * 4u) == 0 &&
           memcmp(a->sid, b->sid, a->n_eff * 4u) == 0 && memcmp(a->tool, b->tool, a->n_eff * 4u) == 0 &&
           memcmp(a->pay, b->pay, a->n_pay * 4u) == 0 && memcmp(a->cnt, b->cnt, a->n_cnt * 4u) == 0;
}

enum { RUN_ALL, RUN_RANGES, RUN_HRT, RUN_NOALLOC_RES, RUN_NOALLOC_HRT, N_RUNS };
static const char *run_name[N_RUNS] = {"resident", "resident over ragged ranges", "host round trip",
                                       "allocation-free resident", "allocation-free host round trip"};

static void run_shape(const Shape *s) {
    const uint32_t C = s->n_cohorts, W = s->W, R = s->R, T = s->T;
    uint32_t *offsets = malloc((C + 1u) * 4u);
    uint32_t *table = malloc((size_t)R * 16u * 4u);
    uint32_t *cdf = R > 1u ? malloc((R - 1u) * 4u) : NULL;
    uint32_t c, k, N, ld;
    size_t i;
    Host in, want, got;
    rc_cohort *h = NULL;
    rc_cohort_desc d;
    rc_buffers b;
    int run;
    const int failures_before = failures;
    printf("shape %s: W=%u R=%u C=%u T=%u\n", s->name, W, R, C, T);
    fflush(stdout);
    offsets[0] = 0u;
    for (c = 0; c < C; ++c) offsets[c + 1u] = offsets[c] + s->size_cycle[c % s->n_cycle];
    N = offsets[C];
    ld = N + 7u; /* padding columns, checked untouched */
    for (i = 0; i < (size_t)R * 16u; ++i) table[i] = next_u32();
    if (cdf) {
        /* Zipf(1.1) thresholds, floor(2^32 * P(route <= k)), in double precision */
        double total = 0.0, acc = 0.0, v;
        for (k = 0; k < R; ++k) total += pow((double)(k + 1u), -1.1);
        for (k = 0; k + 1u < R; ++k) {
            acc += pow((double)(k + 1u), -1.1);
            v = floor(acc / total * 4294967296.0);
            cdf[k] = v >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)v;
        }
    }
    memset(&in, 0, sizeof in);
    memset(&want, 0, sizeof want);
    memset(&got, 0, sizeof got);
    memset(&b, 0, sizeof b);
    if (!(host_alloc(&in, W, ld, T, C) && host_alloc(&want, W, ld, T, C) && host_alloc(&got, W, ld, T, C))) {
        check(0, s->name, "host allocation");
        goto done;
    }
    for (i = 0; i < in.n_state; ++i) in.state[i] = (i % ld) < N ? next_u32() : 0xA5A5A5A5u;
    for (i = 0; i < in.n_outcome; ++i) in.outcome[i] = i < N ? next_u32() : 0x5A5A5A5Au;

    /* expected: the oracle on host copies */
    memcpy(want.state, in.state, in.n_state * 4u);
    memcpy(want.outcome, in.outcome, in.n_outcome * 4u);
    fill_outputs(&want);
    check(rc_oracle_run_chain(N, W, R, C, offsets, table, s->route_mode, cdf, s->thr, want.state,
                              want.outcome, want.sid, want.tool, want.pay, want.cnt, ld, s->step0, T, 0u,
                              C, NULL) == 0,
          s->name, "oracle run");

    memset(&d, 0, sizeof d);
    d.n_sessions = N;
    d.n_words = W;
    d.n_routes = R;
    d.n_cohorts = C;
    d.cohort_offsets = offsets;
    d.table = table;
    d.route_mode = s->route_mode;
    d.route_cdf = cdf;
    d.decide_thr = s->thr;
    check(rc_cohort_create(&d, 0, &h) == RC_OK, s->name, "create");
    b.ld = ld;
    check(hipMalloc((void **)&b.state, in.n_state * 4u) == hipSuccess &&
              hipMalloc((void **)&b.outcome, in.n_outcome * 4u) == hipSuccess &&
              hipMalloc((void **)&b.eff_sid, in.n_eff * 4u) == hipSuccess &&
              hipMalloc((void **)&b.eff_tool, in.n_eff * 4u) == hipSuccess &&
              hipMalloc((void **)&b.eff_payload, in.n_pay * 4u) == hipSuccess &&
              hipMalloc((void **)&b.n_taken, in.n_cnt * 4u) == hipSuccess,
          s->name, "device allocation");
    if (!h || failures > failures_before) goto done;

    for (run = 0; run < N_RUNS; ++run) {
        uint32_t launches = 0, copies = 0;
        int st = RC_OK;
        check(hipMemcpy(b.state, in.state, in.n_state * 4u, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemcpy(b.outcome, in.outcome, in.n_outcome * 4u, hipMemcpyHostToDevice) == hipSuccess &&
                  hipMemset(b.eff_sid, 0xFF, in.n_eff * 4u) == hipSuccess &&
                  hipMemset(b.eff_tool, 0xFF, in.n_eff * 4u) == hipSuccess &&
                  hipMemset(b.eff_payload, 0xFF, in.n_pay * 4u) == hipSuccess &&
                  hipMemset(b.n_taken, 0xFF, in.n_cnt * 4u) == hipSuccess &&
                  hipDeviceSynchronize() == hipSuccess,
              s->name, "upload");
        switch (run) {
            case RUN_ALL:
                st = rc_cohort_run_chain(h, &b, s->step0, T, RC_MODE_RESIDENT, 0u, C, NULL);
                break;
            case RUN_RANGES: {
                /* three ragged ranges, last first */
                const uint32_t c1 = C / 3u, c2 = (2u * C) / 3u + (C > 2u ? 1u : 0u);
                const uint32_t lo[3] = {c2 < C ? c2 : C, 0u, c1};
                const uint32_t hi[3] = {C, c1, c2 < C ? c2 : C};
                for (k = 0; k < 3u && st == RC_OK; ++k)
                    st = rc_cohort_run_chain(h, &b, s->step0, T, RC_MODE_RESIDENT, lo[k], hi[k], NULL);
                break;
            }
            case RUN_HRT:
                st = rc_cohort_run_chain(h, &b, s->step0, T, RC_MODE_HOST_ROUNDTRIP, 0u, C, NULL);
                break;
            case RUN_NOALLOC_RES:
                st = rc_cohort_run_chain_noalloc(h, &b, s->step0, T, RC_MODE_RESIDENT, 0u, C, NULL);
                break;
            default:
                st = rc_cohort_run_chain_noalloc(h, &b, s->step0, T, RC_MODE_HOST_ROUNDTRIP, 0u, C, NULL);
                break;
        }
        check(st == RC_OK, run_name[run], rc_status_string(st));
        check(hipDeviceSynchronize() == hipSuccess, run_name[run], "synchronize");
        check(rc_cohort_last_counts(h, &launches, &copies) == RC_OK, run_name[run], "last counts");
        if (run == RUN_ALL || run == RUN_NOALLOC_RES)
            check(launches == 1u && copies == 0u, run_name[run], "one launch and no copy");
        if (run == RUN_HRT || run == RUN_NOALLOC_HRT)
            check(launches >= T + 1u && copies == T, run_name[run], "T copies and at least T + 1 launches");
        check(hipMemcpy(got.state, b.state, in.n_state * 4u, hipMemcpyDeviceToHost) == hipSuccess &&
                  hipMemcpy(got.outcome, b.outcome, in.n_outcome * 4u, hipMemcpyDeviceToHost) == hipSuccess &&
                  hipMemcpy(got.sid, b.eff_sid, in.n_eff * 4u, hipMemcpyDeviceToHost) == hipSuccess &&
                  hipMemcpy(got.tool, b.eff_tool, in.n_eff * 4u, hipMemcpyDeviceToHost) == hipSuccess &&
                  hipMemcpy(got.pay, b.eff_payload, in.n_pay * 4u, hipMemcpyDeviceToHost) == hipSuccess &&
                  hipMemcpy(got.cnt, b.n_taken, in.n_cnt * 4u, hipMemcpyDeviceToHost) == hipSuccess,
              run_name[run], "download");
        check(same(&got, &want), s->name, run_name[run]);
    }

done:
    if (h) rc_cohort_destroy(h);
    hipFree(b.state);
    hipFree(b.outcome);
    hipFree(b.eff_sid);
    hipFree(b.eff_tool);
    hipFree(b.eff_payload);
    hipFree(b.n_taken);
    host_free(&in);
    host_free(&want);
    host_free(&got);
    free(offsets);
    free(table);
    free(cdf);
}

int main(void) {
    static const uint32_t k256[1] = {256};
    static const uint32_t mixed[7] = {32, 64, 256, 128, 32, 200, 17};
    static const uint32_t k64[1] = {64};
    static const uint32_t k32[1] = {32};
    const Shape shapes[4] = {
        {"two-role split", 32, 256, RC_ROUTE_MOD, 32768, 16, 5u, 300, k256, 1},
        {"table image", 64, 1024, RC_ROUTE_CDF, 3277, 16, 0xFFFFFFF8u, 500, mixed, 7},
        {"pipelined split", 16, 16, RC_ROUTE_MOD, 32768, 8, 0u, 1, k64, 1},
        {"one-lane chain", 8, 4, RC_ROUTE_MOD, 32768, 1, 12345u, 32, k32, 1},
    };
    int i;
    sm_state = 20261202u;
    for (i = 0; i < 4; ++i) run_shape(&shapes[i]);
    if (failures) {
        printf("%d check(s) failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
