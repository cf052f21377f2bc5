// rc_pack.cpp -- the cohort shares of a set of control events (host code of
// the library): fixed-partition eligibility F, the exact offline packing P*
// with a witness schedule, and the local-overlap bound U (the paper's Section
// 3 model under the equal relative deadlines of Section 4).
//
// Per route, on the grouped and sorted release order:
//   F   one pass over the route's releases: runs of equal window index
//       floor((t - origin) / delta) are the fixed buckets.
//   P*  Algorithm 1 of Section 4: D[j] = max(D[j-1], j + max over the valid
//       starts i of D[i-1] - i + 1), the valid starts kept in a monotone
//       deque (start index, value) whose head is the best one; a moving left
//       pointer drops the starts with t_i < t_j - delta; back-pointers give
//       the witness blocks.
//   U   the same-route active count at a release time t_k is
//       c_k = #{releases in [t_k - delta, t_k]}; event i counts when the
//       largest c_k over the releases in [t_i, t_i + delta] reaches K (the
//       count can only rise at a release), a sliding-window maximum with
//       both window ends moving forward.
// All comparisons are inclusive on the integer-nanosecond clock.
//
// The online route compactor (Section 9, "The next systems test") runs its
// frozen policy per route -- routes never interact -- as one forward sweep
// over the route's releases with a FIFO of queued positions: arrivals at or
// before the trigger t_oldest + delta - L are queued first; at the trigger a
// queue of at least K is launched whole, a shorter one sends its oldest event
// to the CPU; a queue that reaches its capacity (>= K) is launched on the
// arrival that filled it.
//
// rc_cohorts_from_batches turns a batch assignment into the cohort layout of
// the transition (sessions grouped by cohort, cohort offsets): each batch is
// cut into ceil(n / max) near-equal cohorts, its events in index order.

#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <new>
#include <vector>

#include "rc_cohort.h"

namespace {

int64_t floor_div(int64_t a, int64_t b) {  // b > 0
    const int64_t q = a / b;
    return (a % b != 0 && a < 0) ? q - 1 : q;
}

struct RouteResult {
    uint64_t fixed = 0, packed = 0, overlap = 0;
};

// One route's slice: releases t[0..n) ascending; ord[p] is the event index
// of position p.  Appends the witness blocks (start, end) in ascending order.
RouteResult pack_route(const int64_t* t, uint64_t n, uint32_t K, int64_t delta, int64_t origin,
                       std::vector<std::pair<uint64_t, uint64_t>>& blocks) {
    RouteResult res;
    // F: runs of equal window index (one division per run: the run ends at
    // the first release at or past the window's end)
    for (uint64_t p = 0; p < n;) {
        const int64_t end = origin + (floor_div(t[p] - origin, delta) + 1) * delta;
        uint64_t q = p + 1;
        while (q < n && t[q] < end) ++q;
        if (q - p >= K) res.fixed += q - p;
        p = q;
    }
    // P*: Algorithm 1 (1-based j, t_j = t[j - 1])
    std::vector<int64_t> D(n + 1, 0);
    std::vector<uint64_t> back(n + 1, 0);
    std::vector<uint64_t> dq_start(n + 1);
    std::vector<int64_t> dq_val(n + 1);
    uint64_t head = 0, tail = 0;  // deque = [head, tail)
    uint64_t left = 1;            // first start with t_start >= t_j - delta
    for (uint64_t j = 1; j <= n; ++j) {
        D[j] = D[j - 1];
        back[j] = 0;
        if (j >= K) {
            const uint64_t i = j - K + 1;
            const int64_t v = D[i - 1] - (int64_t)i + 1;
            while (tail > head && dq_val[tail - 1] < v) --tail;  // smaller tails
            dq_start[tail] = i;
            dq_val[tail] = v;
            ++tail;
        }
        while (t[left - 1] < t[j - 1] - delta) ++left;  // left <= j always
        while (tail > head && dq_start[head] < left) ++head;
        if (tail > head) {
            const int64_t cand = (int64_t)j + dq_val[head];
            if (cand > D[j]) {
                D[j] = cand;
                back[j] = dq_start[head];
            }
        }
    }
    res.packed = (uint64_t)D[n];
    const size_t first = blocks.size();
    for (uint64_t j = n; j > 0;) {
        if (back[j] == 0) {
            --j;
        } else {
            blocks.emplace_back(back[j] - 1, j);  // positions [start - 1, j)
            j = back[j] - 1;
        }
    }
    std::reverse(blocks.begin() + first, blocks.end());
    // U: c_p = ub(t_p) - lb(t_p - delta); window of p = [lb(t_p), ub(t_p + delta))
    std::vector<uint64_t> c(n);
    {
        uint64_t lo = 0, hi = 0;
        for (uint64_t p = 0; p < n; ++p) {
            while (t[lo] < t[p] - delta) ++lo;
            if (hi < p + 1) hi = p + 1;
            while (hi < n && t[hi] <= t[p]) ++hi;
            c[p] = hi - lo;
        }
    }
    {
        std::vector<uint64_t> dq(n);
        uint64_t h = 0, e = 0;   // deque of positions, c decreasing from the head
        uint64_t wlo = 0, whi = 0;  // window [wlo, whi)
        for (uint64_t p = 0; p < n; ++p) {
            while (wlo < n && t[wlo] < t[p]) ++wlo;  // lb(t_p)
            while (whi < n && t[whi] <= t[p] + delta) {
                while (e > h && c[dq[e - 1]] <= c[whi]) --e;
                dq[e++] = whi++;
            }
            while (e > h && dq[h] < wlo) ++h;
            if (e > h && c[dq[h]] >= K) ++res.overlap;
        }
    }
    return res;
}

// Events grouped by route (counting sort, which keeps index order), each
// route's slice then in (release, index) order.
struct Grouped {
    std::vector<uint64_t> start;  // route r occupies [start[r], start[r + 1])
    std::vector<uint32_t> ord;    // event index of each position
    std::vector<int64_t> t;       // release of each position
};

void group_by_route(const int64_t* rel, const uint32_t* route, uint64_t n, uint32_t n_routes,
                    Grouped& g) {
    g.start.assign((size_t)n_routes + 1u, 0u);
    for (uint64_t i = 0; i < n; ++i) ++g.start[route[i] + 1u];
    for (uint32_t r = 0; r < n_routes; ++r) g.start[r + 1u] += g.start[r];
    g.ord.resize(n);
    {
        std::vector<uint64_t> fill(g.start.begin(), g.start.end() - 1);
        for (uint64_t i = 0; i < n; ++i) g.ord[fill[route[i]]++] = (uint32_t)i;
    }
    g.t.resize(n);
    for (uint64_t p = 0; p < n; ++p) g.t[p] = rel[g.ord[p]];
    std::vector<std::pair<int64_t, uint32_t>> tmp;
    for (uint32_t r = 0; r < n_routes; ++r) {
        const uint64_t a = g.start[r], b = g.start[r + 1u];
        // a slice already in release order is in (release, index) order
        if (std::is_sorted(g.t.begin() + a, g.t.begin() + b)) continue;
        tmp.resize(b - a);
        for (uint64_t p = a; p < b; ++p) tmp[p - a] = {g.t[p], g.ord[p]};
        std::sort(tmp.begin(), tmp.end());
        for (uint64_t p = a; p < b; ++p) {
            g.t[p] = tmp[p - a].first;
            g.ord[p] = tmp[p - a].second;
        }
    }
}

// Checks shared by the two event entry points.
int validate_events(const int64_t* rel, const uint32_t* route, uint64_t n,
                    const uint32_t* k_of_route, uint32_t n_routes, int64_t delta) {
    if (n_routes == 0u || !k_of_route || delta < 1 || delta > INT64_MAX / 4) return RC_E_INVALID;
    if (n > 0 && (!rel || !route)) return RC_E_INVALID;
    if (n >= 0xFFFFFFFFull) return RC_E_INVALID;
    for (uint32_t r = 0; r < n_routes; ++r)
        if (k_of_route[r] == 0u) return RC_E_INVALID;
    for (uint64_t i = 0; i < n; ++i) {
        if (route[i] >= n_routes) return RC_E_INVALID;
        // keep t - delta and t + delta representable
        if (rel[i] > INT64_MAX / 4 || rel[i] < INT64_MIN / 4) return RC_E_INVALID;
    }
    return RC_OK;
}

struct OnlineCounts {
    uint64_t accelerated = 0, fb_deadline = 0, fb_capacity = 0, at_capacity = 0;
};

// The frozen online policy on one route's sorted releases t[0..n).
// launch(positions, count, tau) receives the launched queue and its time.
template <class Launch>
void online_route(const int64_t* t, uint64_t n, uint64_t K, int64_t delta, int64_t latency,
                  uint64_t cap, std::vector<uint64_t>& q, OnlineCounts& c, Launch&& launch) {
    q.clear();
    size_t qh = 0;  // queue = q[qh..)
    uint64_t p = 0;
    auto arrive = [&](uint64_t pos) {
        if (q.size() - qh >= cap) {
            ++c.fb_capacity;
            return;
        }
        q.push_back(pos);
        if (q.size() - qh == cap && cap >= K) {
            launch(q.data() + qh, q.size() - qh, t[pos]);
            c.accelerated += q.size() - qh;
            ++c.at_capacity;
            q.clear();
            qh = 0;
        }
    };
    for (;;) {
        if (qh == q.size()) {
            q.clear();
            qh = 0;
            if (p == n) break;
            arrive(p++);
            continue;
        }
        const int64_t tau = t[q[qh]] + delta - latency;
        if (p < n && t[p] <= tau) {
            arrive(p++);
        } else if (q.size() - qh >= K) {
            launch(q.data() + qh, q.size() - qh, tau);
            c.accelerated += q.size() - qh;
            q.clear();
            qh = 0;
        } else {
            ++c.fb_deadline;
            ++qh;
        }
    }
}

}  // namespace

extern "C" int rc_pack_shares(const int64_t* release_ns, const uint32_t* route, uint64_t n_events,
                              const uint32_t* k_of_route, uint32_t n_routes, int64_t delta_ns,
                              int64_t window_origin_ns, uint32_t* batch_of_event, rc_pack_result* out) {
    if (!out || window_origin_ns > INT64_MAX / 4 || window_origin_ns < INT64_MIN / 4)
        return RC_E_INVALID;
    const int st = validate_events(release_ns, route, n_events, k_of_route, n_routes, delta_ns);
    if (st != RC_OK) return st;
    try {
        Grouped g;
        group_by_route(release_ns, route, n_events, n_routes, g);
        rc_pack_result res = {};
        res.n_events = n_events;
        std::vector<std::pair<uint64_t, uint64_t>> blocks;
        if (batch_of_event)
            for (uint64_t i = 0; i < n_events; ++i) batch_of_event[i] = 0xFFFFFFFFu;
        for (uint32_t r = 0; r < n_routes; ++r) {
            const uint64_t a = g.start[r], b = g.start[r + 1u];
            if (a == b) continue;
            blocks.clear();
            const RouteResult rr = pack_route(g.t.data() + a, b - a, k_of_route[r], delta_ns,
                                              window_origin_ns, blocks);
            res.fixed_eligible += rr.fixed;
            res.packed += rr.packed;
            res.overlap_eligible += rr.overlap;
            for (const auto& blk : blocks) {
                if (batch_of_event)
                    for (uint64_t p = blk.first; p < blk.second; ++p)
                        batch_of_event[g.ord[a + p]] = (uint32_t)res.n_batches;
                ++res.n_batches;
            }
        }
        *out = res;
        return RC_OK;
    } catch (const std::bad_alloc&) {
        return RC_E_NOMEM;
    }
}

extern "C" int rc_online_compact(const int64_t* release_ns, const uint32_t* route,
                                 uint64_t n_events, const uint32_t* k_of_route, uint32_t n_routes,
                                 int64_t delta_ns, int64_t latency_ns, uint32_t capacity,
                                 uint32_t* batch_of_event, int64_t* launch_ns,
                                 rc_online_result* out) {
    if (!out || capacity == 0u || latency_ns < 0 || latency_ns > delta_ns) return RC_E_INVALID;
    const int st = validate_events(release_ns, route, n_events, k_of_route, n_routes, delta_ns);
    if (st != RC_OK) return st;
    try {
        Grouped g;
        group_by_route(release_ns, route, n_events, n_routes, g);
        if (batch_of_event)
            for (uint64_t i = 0; i < n_events; ++i) batch_of_event[i] = 0xFFFFFFFFu;
        rc_online_result res = {};
        res.n_events = n_events;
        OnlineCounts c;
        std::vector<uint64_t> q;
        for (uint32_t r = 0; r < n_routes; ++r) {
            const uint64_t a = g.start[r], b = g.start[r + 1u];
            if (a == b) continue;
            online_route(g.t.data() + a, b - a, k_of_route[r], delta_ns, latency_ns, capacity, q, c,
                         [&](const uint64_t* pos, size_t m, int64_t tau) {
                             if (batch_of_event)
                                 for (size_t j = 0; j < m; ++j)
                                     batch_of_event[g.ord[a + pos[j]]] = (uint32_t)res.n_batches;
                             if (launch_ns) launch_ns[res.n_batches] = tau;
                             ++res.n_batches;
                         });
        }
        res.accelerated = c.accelerated;
        res.fallback_deadline = c.fb_deadline;
        res.fallback_capacity = c.fb_capacity;
        res.launched_at_capacity = c.at_capacity;
        *out = res;
        return RC_OK;
    } catch (const std::bad_alloc&) {
        return RC_E_NOMEM;
    }
}

extern "C" int rc_cohorts_from_batches(const uint32_t* batch_of_event, uint64_t n_events,
                                       uint64_t n_batches, uint32_t max_cohort, uint32_t* order,
                                       uint32_t* offsets, uint64_t* n_cohorts) {
    if (!n_cohorts || !order || !offsets || max_cohort == 0u) return RC_E_INVALID;
    if (n_events > 0 && !batch_of_event) return RC_E_INVALID;
    if (n_events >= 0xFFFFFFFFull || n_batches > n_events) return RC_E_INVALID;
    for (uint64_t i = 0; i < n_events; ++i)
        if (batch_of_event[i] != 0xFFFFFFFFu && batch_of_event[i] >= n_batches) return RC_E_INVALID;
    try {
        // counting sort by batch (stable: index order inside a batch)
        std::vector<uint64_t> start(n_batches + 1u, 0u);
        for (uint64_t i = 0; i < n_events; ++i)
            if (batch_of_event[i] != 0xFFFFFFFFu) ++start[batch_of_event[i] + 1u];
        for (uint64_t b = 0; b < n_batches; ++b) start[b + 1u] += start[b];
        {
            std::vector<uint64_t> fill(start.begin(), start.end() - 1);
            for (uint64_t i = 0; i < n_events; ++i)
                if (batch_of_event[i] != 0xFFFFFFFFu) order[fill[batch_of_event[i]]++] = (uint32_t)i;
        }
        uint64_t c = 0;
        offsets[0] = 0u;
        for (uint64_t b = 0; b < n_batches; ++b) {
            const uint64_t m = start[b + 1u] - start[b];
            if (m == 0) continue;
            const uint64_t pieces = (m + max_cohort - 1u) / max_cohort;
            const uint64_t base = m / pieces, extra = m % pieces;
            uint64_t at = start[b];
            for (uint64_t j = 0; j < pieces; ++j) {
                at += base + (j < extra ? 1u : 0u);
                offsets[++c] = (uint32_t)at;
            }
        }
        *n_cohorts = c;
        return RC_OK;
    } catch (const std::bad_alloc&) {
        return RC_E_NOMEM;
    }
}
