/*
 * A plain C99 client of rc_cohort.h: it compiles the header as C and links
 * against the library, then calls the entry points that need no GPU.
 *   - status strings and the NULL-handle conventions;
 *   - descriptors the library must reject before any device call;
 *   - the launch plan of three cohorts (every session in exactly one lane,
 *     a cohort of at most 64 sessions inside one wavefront);
 *   - the cohort shares of three events on one route, with values worked out
 *     by hand from the definitions of F, P* and U;
 *   - the cut of two batches into cohorts of at most two sessions.
 * Prints "ok" and exits 0 when every check holds; otherwise names the check
 * that failed and exits 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "rc_cohort.h"

static int failures = 0;

static void check(int cond, const char *what) {
    if (!cond) {
        printf("FAILED: %s\n", what);
        ++failures;
    }
}

static void statuses(void) {
    check(strcmp(rc_status_string(RC_OK), "RC_OK") == 0, "status string RC_OK");
    check(strcmp(rc_status_string(RC_E_INVALID), "RC_E_INVALID") == 0, "status string RC_E_INVALID");
    check(strcmp(rc_status_string(RC_E_NOMEM), "RC_E_NOMEM") == 0, "status string RC_E_NOMEM");
    check(strcmp(rc_status_string(RC_E_DEVICE), "RC_E_DEVICE") == 0, "status string RC_E_DEVICE");
    check(rc_status_string(12345) != NULL, "status string of an unknown code");
    check(rc_cohort_destroy(NULL) == RC_OK, "destroy(NULL) is RC_OK");
    check(rc_cohort_last_counts(NULL, NULL, NULL) == RC_E_INVALID, "last_counts(NULL)");
    check(rc_cohort_plan_info(NULL, NULL, NULL, NULL) == RC_E_INVALID, "plan_info(NULL)");
    check(rc_cohort_run_chain(NULL, NULL, 0, 1, RC_MODE_RESIDENT, 0, 1, NULL) == RC_E_INVALID,
          "run_chain(NULL handle)");
}

static void rejected_descriptors(void) {
    uint32_t offsets[3] = {0, 40, 100};
    uint32_t table[16 * 2];
    rc_cohort_desc d;
    rc_cohort *h = (rc_cohort *)&d; /* must stay untouched on error */
    memset(table, 0, sizeof table);
    memset(&d, 0, sizeof d);
    d.n_sessions = 100;
    d.n_words = 3; /* below RC_MIN_WORDS */
    d.n_routes = 2;
    d.n_cohorts = 2;
    d.cohort_offsets = offsets;
    d.table = table;
    d.route_mode = RC_ROUTE_MOD;
    d.decide_thr = 32768;
    check(rc_cohort_create(&d, 0, &h) == RC_E_INVALID, "W below the minimum is rejected");
    d.n_words = RC_MAX_WORDS + 1;
    check(rc_cohort_create(&d, 0, &h) == RC_E_INVALID, "W above the maximum is rejected");
    d.n_words = 8;
    d.decide_thr = 65537;
    check(rc_cohort_create(&d, 0, &h) == RC_E_INVALID, "a threshold above 65536 is rejected");
    d.decide_thr = 32768;
    offsets[1] = 0; /* an empty cohort */
    check(rc_cohort_create(&d, 0, &h) == RC_E_INVALID, "an empty cohort is rejected");
    offsets[1] = 40;
    d.route_mode = RC_ROUTE_CDF; /* R = 2 needs one threshold */
    check(rc_cohort_create(&d, 0, &h) == RC_E_INVALID, "CDF mode without thresholds is rejected");
    d.route_mode = RC_ROUTE_MOD;
    check(rc_cohort_create(NULL, 0, &h) == RC_E_INVALID, "a NULL descriptor is rejected");
    check(rc_cohort_create(&d, 0, NULL) == RC_E_INVALID, "a NULL output is rejected");
    check(h == (rc_cohort *)&d, "the output is left untouched on error");
}

static void plan(void) {
    /* cohorts of 40, 60 and 256 sessions */
    uint32_t offsets[4] = {0, 40, 100, 356};
    uint32_t table[16];
    uint32_t lane_session[1024], lane_cohort[1024], seen[356];
    uint32_t n_lanes = 0, i, c;
    rc_cohort_desc d;
    memset(table, 0, sizeof table);
    memset(&d, 0, sizeof d);
    d.n_sessions = 356;
    d.n_words = 4;
    d.n_routes = 1;
    d.n_cohorts = 3;
    d.cohort_offsets = offsets;
    d.table = table;
    d.route_mode = RC_ROUTE_MOD;
    check(rc_plan_lanes(&d, 256, NULL, NULL, 0, &n_lanes) == RC_OK, "plan size query");
    check(n_lanes > 0 && n_lanes <= 1024 && n_lanes % 256 == 0, "plan lanes are whole workgroups");
    check(rc_plan_lanes(&d, 256, lane_session, lane_cohort, 1024, &n_lanes) == RC_OK, "plan lanes");
    check(rc_plan_lanes(&d, 256, lane_session, lane_cohort, n_lanes - 1, &n_lanes) == RC_E_INVALID,
          "too small a capacity is rejected");
    check(rc_plan_lanes(&d, 100, NULL, NULL, 0, &n_lanes) == RC_E_INVALID,
          "a workgroup size other than 256 or 512 is rejected");
    memset(seen, 0, sizeof seen);
    for (i = 0; i < n_lanes; ++i) {
        const uint32_t s = lane_session[i];
        if (s == 0xFFFFFFFFu) {
            check(lane_cohort[i] == 0xFFFFFFFFu, "an idle lane has no cohort");
            continue;
        }
        check(s < 356, "a lane's session is in range");
        if (s >= 356) continue;
        ++seen[s];
        c = lane_cohort[i];
        check(c < 3 && offsets[c] <= s && s < offsets[c + 1], "a lane's cohort holds its session");
    }
    for (i = 0; i < 356; ++i) check(seen[i] == 1, "every session is in exactly one lane");
    /* the lanes of the two small cohorts lie inside one wavefront each */
    for (c = 0; c < 2; ++c) {
        uint32_t lo = 0xFFFFFFFFu, hi = 0;
        for (i = 0; i < n_lanes; ++i)
            if (lane_cohort[i] == c) {
                if (i < lo) lo = i;
                if (i > hi) hi = i;
            }
        check(lo / 64 == hi / 64, "a cohort of at most 64 sessions stays inside one wavefront");
    }
}

static void shares(void) {
    /* One route, K = 2, delta = 15 ns, releases 0, 10, 20.  Fixed windows
     * [0, 15) and [15, 30) hold 2 and 1 events: F = 2.  A batch needs a
     * launch time inside every member's [t, t + 15]: {0, 10} (at 10..15) or
     * {10, 20} (at 20..25), never all three (20 > 15): P* = 2.  Event 20
     * sees event 10 still active at 20..25, so all three reach K: U = 3. */
    const int64_t release[3] = {0, 10, 20};
    const uint32_t route[3] = {0, 0, 0};
    const uint32_t k_of_route[1] = {2};
    uint32_t batch[3];
    rc_pack_result r;
    int in_batch = 0, i;
    check(rc_pack_shares(release, route, 3, k_of_route, 1, 15, 0, batch, &r) == RC_OK, "pack shares");
    check(r.n_events == 3 && r.fixed_eligible == 2 && r.packed == 2 && r.overlap_eligible == 3 &&
              r.n_batches == 1, "F = 2, P* = 2, U = 3 and one batch");
    for (i = 0; i < 3; ++i) in_batch += batch[i] == 0u;
    check(in_batch == 2 && batch[1] == 0u && (batch[0] == 0xFFFFFFFFu || batch[2] == 0xFFFFFFFFu),
          "the witness batches two neighbours in release order and leaves one event out");
    check(rc_pack_shares(release, route, 3, k_of_route, 1, 0, 0, NULL, &r) == RC_E_INVALID,
          "delta < 1 is rejected");
}

static void cohorts_from_batches(void) {
    /* batch 0 = events {0, 2, 5, 6}, batch 1 = {1, 4}, event 3 left out;
     * cohorts of at most 2: {0, 2}, {5, 6}, {1, 4} */
    const uint32_t batch_of_event[7] = {0, 1, 0, 0xFFFFFFFFu, 1, 0, 0};
    const uint32_t want_order[6] = {0, 2, 5, 6, 1, 4};
    const uint32_t want_offsets[4] = {0, 2, 4, 6};
    uint32_t order[7], offsets[8];
    uint64_t n_cohorts = 0;
    check(rc_cohorts_from_batches(batch_of_event, 7, 2, 2, order, offsets, &n_cohorts) == RC_OK,
          "cohorts from batches");
    check(n_cohorts == 3, "three cohorts");
    check(memcmp(order, want_order, sizeof want_order) == 0, "sessions grouped by cohort, in event order");
    check(memcmp(offsets, want_offsets, sizeof want_offsets) == 0, "cohort offsets");
    check(rc_cohorts_from_batches(batch_of_event, 7, 2, 0, order, offsets, &n_cohorts) == RC_E_INVALID,
          "max_cohort 0 is rejected");
}

int main(void) {
    statuses();
    rejected_descriptors();
    plan();
    shares();
    cohorts_from_batches();
    if (failures) {
        printf("%d check(s) failed\n", failures);
        return 1;
    }
    printf("ok\n");
    return 0;
}
