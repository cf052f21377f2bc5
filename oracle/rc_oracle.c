/*
 * rc_oracle.c -- reference CPU implementation ("the oracle") of the batched
 * ready-cohort control transition.
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
 * CPU-baseline leg of the benchmark are the only code allowed to load this
 * library.  The product path (the HIP library under paper_2608_12123_amd/)
 * shares no source, header, table or helper with this file and never calls
 * it; it must fail loudly rather than fall back to a CPU path.
 *
 * The oracle is deliberately plain: one thread, no SIMD, no blocking, no
 * fusion, no reordering beyond what the definition states.  All arithmetic is
 * on uint32_t, so every product and sum wraps modulo 2^32.
 *
 * What is computed (the paper's unit of work, Abstract and Section 2 "Unit of
 * execution": a transition reads typed state and an available outcome, routes
 * it, updates the state and emits the next effect; Section 7 "Matched
 * mechanisms": a GPU predicate decides between two synthetic route bodies and
 * the decision is chained over H epochs; Section 11 "Mechanism and sampling
 * scope": a route service additionally needs per-event compaction and effect
 * ordering).  This implementation's synthetic instance, per session s of a
 * cohort and per chained step t with step = step0 + t:
 *
 *   route    r = o mod R                     (route mode MOD)
 *            r = #{k < R-1 : cdf[k] <= o}    (route mode CDF)
 *   decide   d = (fmix32(S[0] ^ o ^ step) & 0xFFFF) < thr, on the state
 *            before this step's update
 *   update   for every word w < W:
 *              d = 1: S[w] = S[w] ^ (table[r][w mod 16] * (w + 1))
 *              d = 0: S[w] = rotl(S[w], (r + 1) mod 32) + o
 *   emit     effect (sid = s, tool = table[r][d] mod 8, payload = S[0..3]
 *            after the update), written at the session's slot of a stable
 *            partition of the cohort: taken sessions first, each population
 *            in ascending session id
 *   count    n_taken[t][c] = number of taken sessions of cohort c
 *   chain    the next outcome of s is fmix32(S[0]) (= fmix32(payload[0]))
 *
 * fmix32 is the 32-bit finalizer of Austin Appleby's MurmurHash3
 * (public domain).
 *
 * Layout (structure of arrays, leading dimension ld >= N):
 *   state[w*ld + s], outcome[s], eff_sid[t*ld + slot], eff_tool[t*ld + slot],
 *   eff_payload[(t*ld + slot)*4 + q], n_taken[t*C + c].
 */
#include <stdint.h>
#include <stdlib.h>

#define RC_ORACLE_ROUTE_MOD 0u
#define RC_ORACLE_ROUTE_CDF 1u

/* MurmurHash3 fmix32: xor-shift 16, multiply, xor-shift 13, multiply,
 * xor-shift 16. */
uint32_t rc_oracle_fmix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

/* Rotate left by k mod 32 bits.  A rotation by 0 (mod 32) is the identity;
 * the shift by 32 that a naive formula would make is avoided. */
uint32_t rc_oracle_rotl(uint32_t x, uint32_t k)
{
    k = k % 32u;
    if (k == 0u)
        return x;
    return (x << k) | (x >> (32u - k));
}

/* Route key of an outcome.  MOD: the outcome modulo the number of routes.
 * CDF: the number of thresholds not above the outcome, i.e. route k owns the
 * outcomes in [cdf[k-1], cdf[k]) with cdf[-1] = 0 and cdf[R-1] = 2^32.
 * Written as the plain count, not as a search. */
uint32_t rc_oracle_route(uint32_t o, uint32_t n_routes, uint32_t route_mode,
                         const uint32_t *route_cdf)
{
    uint32_t k, r;
    if (route_mode == RC_ORACLE_ROUTE_MOD)
        return o % n_routes;
    r = 0u;
    for (k = 0u; k + 1u < n_routes; ++k)
        if (route_cdf[k] <= o)
            ++r;
    return r;
}

/* The per-session binary decision (the predicate of Section 7): 1 = taken. */
uint32_t rc_oracle_decide(uint32_t s0, uint32_t o, uint32_t step, uint32_t thr)
{
    uint32_t h = rc_oracle_fmix32(s0 ^ o ^ step);
    return (h & 0xFFFFu) < thr ? 1u : 0u;
}

/* One state word after the route body selected by d. */
uint32_t rc_oracle_update_word(uint32_t x, uint32_t w, uint32_t r, uint32_t d,
                               uint32_t o, const uint32_t *table)
{
    if (d)
        return x ^ (table[r * 16u + (w % 16u)] * (w + 1u));
    return rc_oracle_rotl(x, r + 1u) + o;
}

/* Argument checks shared by nothing but this file.  Returns 0 when valid. */
static int check_args(uint32_t n_sessions, uint32_t n_words, uint32_t n_routes,
                      uint32_t n_cohorts, const uint32_t *cohort_offsets,
                      const uint32_t *table, uint32_t route_mode,
                      const uint32_t *route_cdf, uint32_t decide_thr,
                      uint32_t ld, uint32_t cohort_begin, uint32_t cohort_end)
{
    uint32_t c;
    if (n_sessions == 0u || n_words < 4u || n_routes == 0u || n_cohorts == 0u)
        return 1;
    if (!cohort_offsets || !table || ld < n_sessions || decide_thr > 65536u)
        return 1;
    if (route_mode != RC_ORACLE_ROUTE_MOD && route_mode != RC_ORACLE_ROUTE_CDF)
        return 1;
    if (route_mode == RC_ORACLE_ROUTE_CDF && n_routes > 1u && !route_cdf)
        return 1;
    if (cohort_offsets[0] != 0u || cohort_offsets[n_cohorts] != n_sessions)
        return 1;
    for (c = 0u; c < n_cohorts; ++c)
        if (cohort_offsets[c + 1u] <= cohort_offsets[c])
            return 1;
    if (cohort_begin > cohort_end || cohort_end > n_cohorts)
        return 1;
    return 0;
}

/*
 * Decision bitmaps ([T][dwords] uint32, dwords = ceil(ld / 32)): bit s mod 32
 * of word [t][s / 32] is the decision of session s at chained step t.
 */
static uint32_t bit_of(const uint32_t *bits, uint32_t dwords, uint32_t t,
                       uint32_t s)
{
    return (bits[(size_t)t * dwords + s / 32u] >> (s % 32u)) & 1u;
}

/*
 * The chain.  With `forced` NULL every decision comes from the predicate;
 * otherwise it is read from the bitmap `forced` and no predicate is evaluated
 * (the no-decision floor of Section 7 "Matched mechanisms": the recorded route
 * sequence is replayed without predicate or selection).  When `record` is not
 * NULL the decision of every stepped session is written into that bitmap
 * (bits of unstepped sessions are left as they are).
 */
static int run_core(uint32_t n_sessions, uint32_t n_words, uint32_t n_routes,
                    uint32_t n_cohorts, const uint32_t *cohort_offsets,
                    const uint32_t *table, uint32_t route_mode,
                    const uint32_t *route_cdf, uint32_t decide_thr,
                    const uint32_t *forced, uint32_t *record,
                    uint32_t *state, uint32_t *outcome, uint32_t *eff_sid,
                    uint32_t *eff_tool, uint32_t *eff_payload,
                    uint32_t *n_taken, uint32_t ld, uint32_t step0,
                    uint32_t n_steps, uint32_t cohort_begin,
                    uint32_t cohort_end)
{
    uint32_t t, c, s, w, q;
    uint32_t *route_of, *taken;
    uint32_t max_size = 0u;
    const uint32_t dwords = (ld + 31u) / 32u;

    if (check_args(n_sessions, n_words, n_routes, n_cohorts, cohort_offsets,
                   table, route_mode, route_cdf, decide_thr, ld, cohort_begin,
                   cohort_end))
        return 1;
    for (c = cohort_begin; c < cohort_end; ++c)
        if (cohort_offsets[c + 1u] - cohort_offsets[c] > max_size)
            max_size = cohort_offsets[c + 1u] - cohort_offsets[c];
    if (max_size == 0u || n_steps == 0u)
        return 0;

    route_of = (uint32_t *)malloc(sizeof(uint32_t) * max_size);
    taken = (uint32_t *)malloc(sizeof(uint32_t) * max_size);
    if (!route_of || !taken) {
        free(route_of);
        free(taken);
        return 2;
    }

    for (t = 0u; t < n_steps; ++t) {
        uint32_t step = step0 + t;
        size_t slice = (size_t)t * ld;

        for (c = cohort_begin; c < cohort_end; ++c) {
            uint32_t b = cohort_offsets[c];
            uint32_t e = cohort_offsets[c + 1u];
            uint32_t n1 = 0u, next_taken, next_not;

            /* Route and decide every session from its pre-update state. */
            for (s = b; s < e; ++s) {
                uint32_t o = outcome[s];
                route_of[s - b] = rc_oracle_route(o, n_routes, route_mode,
                                                  route_cdf);
                if (forced)
                    taken[s - b] = bit_of(forced, dwords, t, s);
                else
                    taken[s - b] = rc_oracle_decide(state[s], o, step, decide_thr);
                if (record) {
                    uint32_t *word = &record[(size_t)t * dwords + s / 32u];
                    *word = (*word & ~(1u << (s % 32u))) |
                            (taken[s - b] << (s % 32u));
                }
                n1 += taken[s - b];
            }

            /* Update, emit at the stable-partition slot, chain the outcome.
             * Walking the cohort in ascending session id and handing out
             * slots from two running counters is the stable partition. */
            next_taken = b;
            next_not = b + n1;
            for (s = b; s < e; ++s) {
                uint32_t r = route_of[s - b];
                uint32_t d = taken[s - b];
                uint32_t o = outcome[s];
                uint32_t slot;

                for (w = 0u; w < n_words; ++w) {
                    size_t at = (size_t)w * ld + s;
                    state[at] = rc_oracle_update_word(state[at], w, r, d, o,
                                                      table);
                }
                slot = d ? next_taken++ : next_not++;
                eff_sid[slice + slot] = s;
                eff_tool[slice + slot] = table[r * 16u + d] % 8u;
                for (q = 0u; q < 4u; ++q)
                    eff_payload[((size_t)t * ld + slot) * 4u + q] =
                        state[(size_t)q * ld + s];
                outcome[s] = rc_oracle_fmix32(state[s]);
            }
            n_taken[(size_t)t * n_cohorts + c] = n1;
        }
    }
    free(route_of);
    free(taken);
    return 0;
}

/*
 * Run T chained steps over the cohorts [cohort_begin, cohort_end).
 * state and outcome are updated in place; effect slices 0..T-1 and
 * n_taken rows 0..T-1 are written.  Sessions of other cohorts and every
 * other element are left untouched.  decisions_out, when not NULL, is a
 * [T][ceil(ld/32)] bitmap that receives every stepped session's decision.
 * Returns 0 on success, 1 on invalid arguments, 2 when scratch memory cannot
 * be allocated.
 */
int rc_oracle_run_chain(uint32_t n_sessions, uint32_t n_words,
                        uint32_t n_routes, uint32_t n_cohorts,
                        const uint32_t *cohort_offsets, const uint32_t *table,
                        uint32_t route_mode, const uint32_t *route_cdf,
                        uint32_t decide_thr, uint32_t *state, uint32_t *outcome,
                        uint32_t *eff_sid, uint32_t *eff_tool,
                        uint32_t *eff_payload, uint32_t *n_taken, uint32_t ld,
                        uint32_t step0, uint32_t n_steps,
                        uint32_t cohort_begin, uint32_t cohort_end,
                        uint32_t *decisions_out)
{
    return run_core(n_sessions, n_words, n_routes, n_cohorts, cohort_offsets,
                    table, route_mode, route_cdf, decide_thr, NULL,
                    decisions_out, state, outcome, eff_sid, eff_tool,
                    eff_payload, n_taken, ld, step0, n_steps, cohort_begin,
                    cohort_end);
}

/*
 * The no-decision floor (Section 7 "Matched mechanisms"): the same chain, but
 * the decision of session s at step t is bit s mod 32 of
 * decisions[t][s / 32] ([T][ceil(ld/32)] words) and no predicate is
 * evaluated, so the step number plays no part.  Everything else (routes,
 * updates, compaction, effects, counts, the chained outcome) is as in
 * rc_oracle_run_chain.  Same return codes.
 */
int rc_oracle_run_floor(uint32_t n_sessions, uint32_t n_words,
                        uint32_t n_routes, uint32_t n_cohorts,
                        const uint32_t *cohort_offsets, const uint32_t *table,
                        uint32_t route_mode, const uint32_t *route_cdf,
                        const uint32_t *decisions, uint32_t *state,
                        uint32_t *outcome, uint32_t *eff_sid,
                        uint32_t *eff_tool, uint32_t *eff_payload,
                        uint32_t *n_taken, uint32_t ld, uint32_t n_steps,
                        uint32_t cohort_begin, uint32_t cohort_end)
{
    if (!decisions)
        return 1;
    return run_core(n_sessions, n_words, n_routes, n_cohorts, cohort_offsets,
                    table, route_mode, route_cdf, 0u, decisions, NULL, state,
                    outcome, eff_sid, eff_tool, eff_payload, n_taken, ld, 0u,
                    n_steps, cohort_begin, cohort_end);
}

/* Count, over every one of the 2^32 outcomes o, the sessions that would be
 * taken for a fixed pre-update word s0 and step.  A brute-force probe of the
 * decision rule for the tests; it only calls rc_oracle_decide. */
uint64_t rc_oracle_count_taken_all_outcomes(uint32_t s0, uint32_t step,
                                            uint32_t thr)
{
    uint64_t n = 0u;
    uint64_t o;
    for (o = 0u; o <= 0xFFFFFFFFull; ++o)
        n += rc_oracle_decide(s0, (uint32_t)o, step, thr);
    return n;
}

/* Count, over every outcome in [lo, hi), how many land on each route.
 * counts must hold n_routes entries and is overwritten. */
void rc_oracle_route_histogram(uint64_t lo, uint64_t hi, uint32_t n_routes,
                               uint32_t route_mode, const uint32_t *route_cdf,
                               uint64_t *counts)
{
    uint64_t o;
    uint32_t r;
    for (r = 0u; r < n_routes; ++r)
        counts[r] = 0u;
    for (o = lo; o < hi; ++o)
        counts[rc_oracle_route((uint32_t)o, n_routes, route_mode,
                               route_cdf)] += 1u;
}
