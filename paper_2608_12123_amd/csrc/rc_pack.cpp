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
    // F: runs of equal window index
    for (uint64_t p = 0; p < n;) {
        const int64_t w = floor_div(t[p] - origin, delta);
        uint64_t q = p + 1;
        while (q < n && floor_div(t[q] - origin, delta) == w) ++q;
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

}  // namespace

extern "C" int rc_pack_shares(const int64_t* release_ns, const uint32_t* route, uint64_t n_events,
                              const uint32_t* k_of_route, uint32_t n_routes, int64_t delta_ns,
                              int64_t window_origin_ns, uint32_t* batch_of_event, rc_pack_result* out) {
    if (!out || n_routes == 0u || !k_of_route || delta_ns < 1) return RC_E_INVALID;
    if (n_events > 0 && (!release_ns || !route)) return RC_E_INVALID;
    if (n_events >= 0xFFFFFFFFull) return RC_E_INVALID;
    for (uint32_t r = 0; r < n_routes; ++r)
        if (k_of_route[r] == 0u) return RC_E_INVALID;
    for (uint64_t i = 0; i < n_events; ++i) {
        if (route[i] >= n_routes) return RC_E_INVALID;
        // keep t - delta and t + delta representable
        if (release_ns[i] > INT64_MAX / 4 || release_ns[i] < INT64_MIN / 4) return RC_E_INVALID;
    }
    if (delta_ns > INT64_MAX / 4) return RC_E_INVALID;
    try {
        // grouped order: by route (counting sort), then release, then index
        std::vector<uint64_t> start((size_t)n_routes + 1u, 0u);
        for (uint64_t i = 0; i < n_events; ++i) ++start[route[i] + 1u];
        for (uint32_t r = 0; r < n_routes; ++r) start[r + 1u] += start[r];
        std::vector<uint32_t> ord(n_events);
        {
            std::vector<uint64_t> fill(start.begin(), start.end() - 1);
            for (uint64_t i = 0; i < n_events; ++i) ord[fill[route[i]]++] = (uint32_t)i;
        }
        std::vector<int64_t> t(n_events);
        rc_pack_result res = {};
        res.n_events = n_events;
        std::vector<std::pair<uint64_t, uint64_t>> blocks;
        if (batch_of_event)
            for (uint64_t i = 0; i < n_events; ++i) batch_of_event[i] = 0xFFFFFFFFu;
        for (uint64_t p = 0; p < n_events; ++p) t[p] = release_ns[ord[p]];
        std::vector<std::pair<int64_t, uint32_t>> tmp;
        for (uint32_t r = 0; r < n_routes; ++r) {
            const uint64_t a = start[r], b = start[r + 1u];
            if (a == b) continue;
            // the counting sort kept index order, so a slice already in
            // release order is in (release, index) order
            if (!std::is_sorted(t.begin() + a, t.begin() + b)) {
                tmp.resize(b - a);
                for (uint64_t p = a; p < b; ++p) tmp[p - a] = {t[p], ord[p]};
                std::sort(tmp.begin(), tmp.end());
                for (uint64_t p = a; p < b; ++p) {
                    t[p] = tmp[p - a].first;
                    ord[p] = tmp[p - a].second;
                }
            }
            blocks.clear();
            const RouteResult rr = pack_route(t.data() + a, b - a, k_of_route[r], delta_ns,
                                              window_origin_ns, blocks);
            res.fixed_eligible += rr.fixed;
            res.packed += rr.packed;
            res.overlap_eligible += rr.overlap;
            for (const auto& blk : blocks) {
                if (batch_of_event)
                    for (uint64_t p = blk.first; p < blk.second; ++p)
                        batch_of_event[ord[a + p]] = (uint32_t)res.n_batches;
                ++res.n_batches;
            }
        }
        *out = res;
        return RC_OK;
    } catch (const std::bad_alloc&) {
        return RC_E_NOMEM;
    }
}
