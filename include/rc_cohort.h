/*
 * rc_cohort.h -- C ABI of the batched ready-cohort control transition,
 * implemented with hand-written HIP kernels for AMD Instinct MI355X (gfx950).
 *
 * What the library computes.  A session holds W uint32 state words and one
 * pending outcome.  Sessions are grouped into cohorts (contiguous session
 * ranges of at most 256).  One chained step of a cohort applies the paper's
 * unit of control work to every member (Abstract; Section 2 "Unit of
 * execution": read typed state and an available outcome, route it, update the
 * state, emit the next effect) with the decision made on the GPU (Section 7
 * "Matched mechanisms": a GPU predicate selects one of two route bodies), and
 * orders the emitted effects by a per-cohort compaction (Section 11
 * "Mechanism and sampling scope" names per-event compaction and effect
 * ordering as what a route service still needs).  Per session s, at step
 * number `step`, with o its pending outcome and all arithmetic modulo 2^32:
 *
 *   route   r = o mod R                          (RC_ROUTE_MOD)
 *           r = #{k < R-1 : route_cdf[k] <= o}   (RC_ROUTE_CDF)
 *   decide  d = (fmix32(S[0] ^ o ^ step) & 0xFFFF) < decide_thr, on the
 *           state before the update; fmix32 is MurmurHash3's finalizer
 *   update  d = 1: S[w] ^= table[r][w mod 16] * (w + 1)       for all w < W
 *           d = 0: S[w]  = rotl(S[w], (r + 1) mod 32) + o     for all w < W
 *   emit    effect (sid = s, tool = table[r][d] mod 8, payload = S[0..3]
 *           after the update) at the session's slot of the stable partition
 *           of its cohort: taken sessions first, each group in ascending sid
 *   count   n_taken[t][c] = taken sessions of cohort c at chained step t
 *   chain   the session's next outcome is fmix32(S[0])
 *
 * Chaining T steps with the decision kept on the device (RC_MODE_RESIDENT)
 * is the device-resident mechanism of Section 7; RC_MODE_HOST_ROUNDTRIP
 * copies a 4-byte decision word to the host after every step and lets the
 * host select and launch the route-body kernels (the host round trip of
 * Section 7).  Both produce bit-identical outputs.
 *
 * Conventions.  All functions are extern "C", return an rc_status and never
 * throw or abort.  RC_E_INVALID is detected on the host before anything is
 * enqueued, so no caller buffer is touched.  After RC_E_DEVICE the contents
 * of the output buffers are unspecified, but the handle stays valid and can
 * be destroyed.  A handle must not be used by two threads at once.
 */
#ifndef RC_COHORT_H
#define RC_COHORT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rc_cohort rc_cohort; /* opaque; owned by the library */

enum rc_status {
    RC_OK = 0,
    RC_E_INVALID = 1, /* bad argument; detected before any GPU work        */
    RC_E_NOMEM = 2,   /* host or device allocation failed                 */
    RC_E_DEVICE = 3   /* no usable gfx950 device, or a HIP call failed      */
};

enum rc_route_mode {
    RC_ROUTE_MOD = 0, /* r = o mod R                                       */
    RC_ROUTE_CDF = 1  /* r = number of route_cdf thresholds <= o            */
};

enum rc_chain_mode {
    RC_MODE_RESIDENT = 0,      /* one launch; decisions never leave the GPU */
    RC_MODE_HOST_ROUNDTRIP = 1 /* per step: decide kernel, 4-byte copy to
                                  pinned host memory, stream sync, host
                                  launches the selected body kernels        */
};

#define RC_MIN_WORDS 4u      /* the payload needs words 0..3 */
#define RC_MAX_WORDS 64u
#define RC_MAX_ROUTES 1024u
#define RC_MAX_COHORT 256u
#define RC_MAX_SESSIONS (1u << 28)
#define RC_NOALLOC_MAX_SESSIONS (1u << 20) /* rc_cohort_run_chain_noalloc */

/*
 * Problem description (the paper's problem statement: sessions with typed
 * state, route keys derived from outcomes, cohorts of size K; Sections 2-3).
 * Every pointer is HOST memory read only during rc_cohort_create; the
 * library copies what it needs and the caller keeps ownership.
 */
typedef struct rc_cohort_desc {
    uint32_t n_sessions;            /* N, 1 <= N <= RC_MAX_SESSIONS          */
    uint32_t n_words;               /* W, RC_MIN_WORDS <= W <= RC_MAX_WORDS   */
    uint32_t n_routes;              /* R, 1 <= R <= RC_MAX_ROUTES             */
    uint32_t n_cohorts;             /* C >= 1                                 */
    const uint32_t *cohort_offsets; /* [C+1]: 0 = b_0 < b_1 < ... < b_C = N;
                                       cohort c is sessions [b_c, b_{c+1}),
                                       of size 1..RC_MAX_COHORT              */
    const uint32_t *table;          /* [R][16] row-major transition table    */
    uint32_t route_mode;            /* enum rc_route_mode                     */
    const uint32_t *route_cdf;      /* [R-1] nondecreasing thresholds in CDF
                                       mode (may be NULL when R == 1);
                                       ignored in MOD mode                   */
    uint32_t decide_thr;            /* 0..65536; 0 = never taken,
                                       65536 = always taken                  */
} rc_cohort_desc;

/*
 * Caller-owned DEVICE buffers on the handle's device, structure of arrays
 * with leading dimension ld >= N.  For a call that runs T steps:
 *   state        [W][ld]     in/out  word w of session s at state[w*ld + s]
 *   outcome      [ld]        in/out  pending outcome; on return the outcome
 *                                    for the step after the last one
 *   eff_sid      [T][ld]     out     effect slice t, slot j at [t*ld + j]
 *   eff_tool     [T][ld]     out
 *   eff_payload  [T][ld][4]  out     payload word q at [(t*ld + j)*4 + q]
 *                                    (16 contiguous bytes per effect)
 *   n_taken      [T][C]      out     at [t*C + c]
 * Effect slice t of a call is written at the slice offsets above relative
 * to the pointers passed; a caller chaining several calls into one log
 * passes pointers advanced by the slices already written.  The six buffers
 * must not overlap (checked).  Only the sessions, effect slots and n_taken
 * entries of the cohorts in [cohort_begin, cohort_end) are written; every
 * other element, including the padding columns [N, ld), stays unchanged.
 */
typedef struct rc_buffers {
    uint32_t *state;
    uint32_t *outcome;
    uint32_t *eff_sid;
    uint32_t *eff_tool;
    uint32_t *eff_payload;
    uint32_t *n_taken;
    uint32_t ld;
} rc_buffers;

/*
 * Validate `desc`, then bind to HIP device `hip_device` (an ordinal), copy
 * the cohort offsets, table and thresholds to device memory the library
 * owns, and build the launch plan (which cohorts share a workgroup).
 * Writes the new handle to *out (left untouched on error).
 * Errors: RC_E_INVALID for a bad descriptor or out == NULL (checked before
 * any device call); RC_E_DEVICE when the device does not exist or is not a
 * gfx950; RC_E_NOMEM when an allocation fails.
 */
int rc_cohort_create(const rc_cohort_desc *desc, int hip_device, rc_cohort **out);

/*
 * One step (T = 1) of the cohorts [cohort_begin, cohort_end) with step
 * number `step`, in resident mode: exactly rc_cohort_run_chain(h, b, step,
 * 1, RC_MODE_RESIDENT, cohort_begin, cohort_end, hip_stream).
 */
int rc_cohort_step(rc_cohort *h, const rc_buffers *b, uint32_t step,
                   uint32_t cohort_begin, uint32_t cohort_end, void *hip_stream);

/*
 * n_steps chained steps of the cohorts [cohort_begin, cohort_end); step t
 * (0-based) uses the step number step0 + t (mod 2^32).  `hip_stream` is a
 * hipStream_t of the handle's device (NULL = the null stream).
 * RC_MODE_RESIDENT enqueues one kernel launch and returns without waiting.
 * RC_MODE_HOST_ROUNDTRIP synchronizes the stream once per step (that
 * observation is the mechanism being measured) and returns after enqueuing
 * the last body kernel.  Its per-step scratch (a slot permutation and two
 * counter words) belongs to the handle; a host-round-trip call first makes
 * its stream wait for the previous host-round-trip call on the same handle
 * (an event the handle records after that call's last body kernel), so
 * calls on different streams never share the scratch.  n_steps == 0 or an
 * empty cohort range is a no-op.  Chains compose: (T1 steps from step0)
 * then (T2 steps from step0 + T1) equals T1 + T2 steps from step0.
 * Buffer checks: the six buffers must lie inside HIP allocations of the
 * handle's device, each inside one.  The check sees allocations as the HIP
 * runtime made them, so a buffer carved out of a larger allocation (a block
 * of a caching allocator, say) passes whenever it stays inside that
 * allocation: sizing each buffer for its extent is the caller's part.  The
 * handle remembers the last 16 buffer sets (pointers and extents) that
 * passed and does not query the runtime again for them.
 * Errors: RC_E_INVALID for a NULL handle/buffer, ld < N, a bad range or
 * mode, overlapping buffers, or a buffer outside the allocations of the
 * handle's device; RC_E_DEVICE when a launch or copy fails.
 */
int rc_cohort_run_chain(rc_cohort *h, const rc_buffers *b, uint32_t step0,
                        uint32_t n_steps, int mode, uint32_t cohort_begin,
                        uint32_t cohort_end, void *hip_stream);

/*
 * The no-decision floor (Section 7 "Matched mechanisms": the recorded route
 * sequence replayed with no predicate and no selection; a structural floor
 * for the two mechanisms above, not an admissible online policy).  It is the
 * resident chain of n_steps steps with one change: the decision of session s
 * at chained step t is read from `decisions` instead of computed by the
 * predicate, so no step number is involved.  Routes, updates, the
 * stable-partition compaction, effects, taken counts and the chained
 * outcome are computed exactly as in rc_cohort_run_chain; given the
 * decisions that rc_cohort_run_chain(step0, ...) makes on the same inputs,
 * the outputs are bit-identical to it.
 *   decisions  caller-owned DEVICE memory of the handle's device, read only:
 *              [n_steps][dwords] uint32 with dwords = ceil(b->ld / 32); bit
 *              (s mod 32) of word [t][s / 32] is session s's decision at
 *              step t (1 = taken).  Bits of sessions outside the stepped
 *              cohorts are ignored.  It must not overlap any buffer of `b`.
 * One kernel launch, enqueued on `hip_stream`; returns without waiting.
 * n_steps == 0 or an empty cohort range is a no-op.  Errors: those of
 * rc_cohort_run_chain, and RC_E_INVALID when `decisions` is NULL, overlaps a
 * buffer, or does not lie with its whole extent inside one HIP allocation of
 * the handle's device (the same check as the six buffers': sizing it is the
 * caller's part).
 */
int rc_cohort_run_floor(rc_cohort *h, const rc_buffers *b, const uint32_t *decisions,
                        uint32_t n_steps, uint32_t cohort_begin, uint32_t cohort_end,
                        void *hip_stream);

/*
 * For callers that cannot allocate device memory while they run: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc.  Exactly rc_cohort_run_chain (same arguments, same outputs),
 * except that in RC_MODE_HOST_ROUNDTRIP the per-step scratch -- the
 * permutation of the stepped sessions and the two counter words -- lives in
 * one fixed array of device memory of the library (4 MiB plus 256 bytes per
 * device, held until the process ends) instead of the handle's buffers, and
 * the counter words are cleared by a kernel launch (no memset) at the start
 * of every call.  The call allocates nothing: no hipMalloc, hipFree or
 * allocating library routine (RC_MODE_RESIDENT never uses scratch).  All
 * host-round-trip calls of this entry point on one device share the array:
 * each waits on its stream for the previous one (an event recorded after its
 * last body kernel), which orders calls made from one host thread; calls
 * made from several host threads at once race.
 * Errors: those of rc_cohort_run_chain, and RC_E_INVALID (before anything is
 * enqueued) when the stepped cohorts hold more than RC_NOALLOC_MAX_SESSIONS
 * sessions.
 */
int rc_cohort_run_chain_noalloc(rc_cohort *h, const rc_buffers *b, uint32_t step0,
                                uint32_t n_steps, int mode, uint32_t cohort_begin,
                                uint32_t cohort_end, void *hip_stream);

/* Release the handle's device and host resources.  Waits for nothing: the
 * caller synchronizes its streams first.  rc_cohort_destroy(NULL) is RC_OK. */
int rc_cohort_destroy(rc_cohort *h);

/* Static, NUL-terminated name of a status code ("RC_OK", ...). */
const char *rc_status_string(int status);

/*
 * Kernel launches and device-to-host copies enqueued by the last successful
 * rc_cohort_run_chain / rc_cohort_step / rc_cohort_run_floor on this handle
 * (resident and floor: 1 and 0; host round trip: at least T + 1 launches
 * and exactly T copies).  Either output pointer may be NULL.  RC_E_INVALID
 * when h is NULL.
 */
int rc_cohort_last_counts(const rc_cohort *h, uint32_t *launches, uint32_t *d2h_copies);

/*
 * Launch-plan summary: workgroups in the plan, lanes per workgroup, and
 * lanes left idle by packing (cohorts never straddle a workgroup, and a
 * cohort of at most 64 sessions never straddles a wavefront).  Any output
 * pointer may be NULL.  RC_E_INVALID when h is NULL.
 */
int rc_cohort_plan_info(const rc_cohort *h, uint32_t *n_workgroups,
                        uint32_t *lanes_per_workgroup, uint32_t *idle_lanes);

/*
 * Host-only inspection of the launch plan the library would build for
 * `desc` with workgroups of `lanes_per_workgroup` lanes (256 or 512; the
 * library picks one of these per handle).  No device is used.  Writes
 * *n_lanes = bins * lanes_per_workgroup.  When both arrays are non-NULL
 * (capacity >= *n_lanes entries each, host memory) it also writes, for every
 * plan lane, the session it processes and that session's cohort, derived
 * exactly as the kernels derive them (0xFFFFFFFF for idle lanes).  Every
 * session appears in exactly one lane.  Errors: RC_E_INVALID for a bad
 * descriptor, lane count, NULL n_lanes or too small a capacity.
 */
int rc_plan_lanes(const rc_cohort_desc *desc, uint32_t lanes_per_workgroup,
                  uint32_t *lane_session, uint32_t *lane_cohort, uint32_t capacity,
                  uint32_t *n_lanes);

/*
 * Cohort shares of a set of control events (host only; no device is used).
 * The paper's model (Section 3 "Events and the hardware threshold" and "Four
 * shares"): event i has an integer-nanosecond release t_i, a latest launch
 * t_i + delta (the equal relative deadlines of Section 4) and a route r_i; a
 * batch is feasible when its events share a route, number at least K_r, and
 * admit a launch time inside every member's [t_i, t_i + delta]
 * (Eq. feasible-batch; comparisons inclusive).  Returned numerators (divide
 * by n_events for the shares):
 *   fixed_eligible    F:  events in buckets (origin-aligned half-open window
 *                     [origin + k delta, origin + (k+1) delta), route) of at
 *                     least K_r events (Eq. fixed);
 *   packed            P*: the largest number of events covered by disjoint
 *                     feasible batches (Eq. dp, Algorithm 1: grouped sort,
 *                     moving left pointer, monotone deque), exact;
 *   overlap_eligible  U:  events whose route's active count reaches K_r at
 *                     some launch time inside their own interval (Eq. upper);
 *   n_batches         batches of the returned witness schedule.
 * F <= P* <= U always (Proposition "Boundary ordering").
 *   release_ns, route  HOST arrays of n_events; route[i] < n_routes.
 *   k_of_route         HOST array of n_routes thresholds, each >= 1.
 *   delta_ns           >= 1; |release|, delta, |window_origin_ns| at most
 *                      INT64_MAX / 4.
 *   batch_of_event     optional HOST array of n_events (NULL: not written):
 *                      the witness, the batch of every event or 0xFFFFFFFF
 *                      for events left out; batches are numbered by route,
 *                      then by first release, and each is a contiguous run
 *                      of the route's release order (Section 4, "Contiguous
 *                      block form").
 * Errors: RC_E_INVALID for a NULL required pointer, a route out of range, a
 * zero threshold, delta < 1, a clock value out of range or
 * n_events >= 2^32 - 1 (nothing written); RC_E_NOMEM when host memory runs
 * out.
 */
typedef struct {
    uint64_t n_events;
    uint64_t fixed_eligible;   /* numerator of F  */
    uint64_t packed;           /* numerator of P* */
    uint64_t overlap_eligible; /* numerator of U  */
    uint64_t n_batches;
} rc_pack_result;

int rc_pack_shares(const int64_t *release_ns, const uint32_t *route, uint64_t n_events,
                   const uint32_t *k_of_route, uint32_t n_routes, int64_t delta_ns,
                   int64_t window_origin_ns, uint32_t *batch_of_event, rc_pack_result *out);

/*
 * Online route compactor (host only): the runtime of Section 9 ("The next
 * systems test") under one frozen policy, and its achieved share A (the
 * share of events it accelerates; R_A = (A - F) / (P* - F), Eq.
 * online-recovery).  Events (same arguments and limits as rc_pack_shares)
 * arrive in release order into a FIFO queue of their route.  A launch at
 * host time tau starts on the device at tau + latency_ns, which must be no
 * later than every member's deadline t_i + delta_ns.  The policy:
 *   - a queue's trigger is t_oldest + delta - latency; arrivals at or before
 *     it are queued first;
 *   - at the trigger, a queue of at least K_r events is launched whole; a
 *     shorter one sends its oldest event to the CPU (fallback_deadline);
 *   - a queue that reaches `capacity` events (>= K_r) is launched at the
 *     arrival that filled it (launched_at_capacity); with capacity < K_r an
 *     arrival that finds its queue full goes to the CPU (fallback_capacity).
 * Every launched batch is feasible in the sense of Eq. feasible-batch, so
 * accelerated <= packed of rc_pack_shares on the same events.
 *   latency_ns      0 <= latency_ns <= delta_ns.
 *   capacity        queue capacity per route, >= 1 (0xFFFFFFFF: unlimited).
 *   batch_of_event  optional HOST array of n_events: the launched batch of
 *                   every event, 0xFFFFFFFF for the CPU; batches numbered by
 *                   route, then launch order.
 *   launch_ns       optional HOST array with room for n_events entries: the
 *                   launch time of every batch (first n_batches written).
 * Errors: as rc_pack_shares, and RC_E_INVALID for capacity 0 or a latency
 * outside [0, delta_ns].
 */
typedef struct {
    uint64_t n_events;
    uint64_t accelerated;          /* numerator of A */
    uint64_t fallback_deadline;
    uint64_t fallback_capacity;
    uint64_t n_batches;
    uint64_t launched_at_capacity; /* batches launched because their queue was full */
} rc_online_result;

int rc_online_compact(const int64_t *release_ns, const uint32_t *route, uint64_t n_events,
                      const uint32_t *k_of_route, uint32_t n_routes, int64_t delta_ns,
                      int64_t latency_ns, uint32_t capacity, uint32_t *batch_of_event,
                      int64_t *launch_ns, rc_online_result *out);

/*
 * Cohorts of the transition from a batch assignment (host only), so that the
 * batches of rc_pack_shares or rc_online_compact can be fed to
 * rc_cohort_create / rc_cohort_run_chain.  Each batch of n events is cut into
 * ceil(n / max_cohort) cohorts of near-equal size (the first n mod pieces
 * one larger), its events in index order; events with batch 0xFFFFFFFF are
 * left out.
 *   batch_of_event  HOST array of n_events; entries < n_batches or 0xFFFFFFFF.
 *   max_cohort      >= 1 (the transition takes cohorts of at most 256).
 *   order           HOST array with room for n_events: the event index of
 *                   every session, sessions grouped by cohort, cohorts by
 *                   batch.
 *   offsets         HOST array with room for n_events + 1: cohort c holds
 *                   sessions [offsets[c], offsets[c + 1]); offsets[0] = 0.
 *   n_cohorts       out: the number of cohorts.
 * Errors: RC_E_INVALID for a NULL pointer, max_cohort 0, n_batches >
 * n_events, a batch id out of range or n_events >= 2^32 - 1 (nothing
 * written); RC_E_NOMEM when host memory runs out.
 */
int rc_cohorts_from_batches(const uint32_t *batch_of_event, uint64_t n_events, uint64_t n_batches,
                            uint32_t max_cohort, uint32_t *order, uint32_t *offsets,
                            uint64_t *n_cohorts);

#ifdef __cplusplus
}
#endif

#endif /* RC_COHORT_H */
