// rc_host.cpp -- host-only part of the ready-cohort library: descriptor
// validation, the launch plan (which cohorts share a workgroup, and how a
// cohort range maps to bins) and the entry points that need no device.
// Plain C++17; the HIP part (rc_cohort.hip) and a sanitizer build of the
// host code both compile it.
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "rc_plan.h"

namespace rc_plan {

int validate_desc(const rc_cohort_desc* d) {
    if (!d) return RC_E_INVALID;
    if (d->n_sessions < 1u || d->n_sessions > RC_MAX_SESSIONS) return RC_E_INVALID;
    if (d->n_words < RC_MIN_WORDS || d->n_words > RC_MAX_WORDS) return RC_E_INVALID;
    if (d->n_routes < 1u || d->n_routes > RC_MAX_ROUTES) return RC_E_INVALID;
    if (d->n_cohorts < 1u || d->n_cohorts > d->n_sessions) return RC_E_INVALID;
    if (!d->cohort_offsets || !d->table) return RC_E_INVALID;
    if (d->route_mode != RC_ROUTE_MOD && d->route_mode != RC_ROUTE_CDF) return RC_E_INVALID;
    if (d->decide_thr > 65536u) return RC_E_INVALID;
    const uint32_t* off = d->cohort_offsets;
    if (off[0] != 0u || off[d->n_cohorts] != d->n_sessions) return RC_E_INVALID;
    for (uint32_t c = 0; c < d->n_cohorts; ++c) {
        if (off[c + 1] <= off[c]) return RC_E_INVALID;
        if (off[c + 1] - off[c] > RC_MAX_COHORT) return RC_E_INVALID;
    }
    if (d->route_mode == RC_ROUTE_CDF && d->n_routes > 1u) {
        if (!d->route_cdf) return RC_E_INVALID;
        for (uint32_t k = 1; k + 1u < d->n_routes; ++k)
            if (d->route_cdf[k] < d->route_cdf[k - 1]) return RC_E_INVALID;
    }
    return RC_OK;
}

// Pack cohorts into bins of nw wavefronts; a bin is one workgroup.  First
// every cohort of at most 64 sessions, in order, each into the first
// wavefront of the open bin with room for it (at most WD_MAXC cohorts per
// wavefront; such a cohort never straddles a wavefront), then the larger
// ones, each starting on a wavefront boundary and spanning whole
// wavefronts.  No cohort straddles a bin.  A cohort never goes to an
// earlier bin than the one before it, except that a large cohort may fill
// the free wavefronts of the bin before the open one, so the bins of a
// cohort range are contiguous up to one bin on each side.
void build_plan(const uint32_t* off, uint32_t C, uint32_t nw_per_bin, Plan& P) {
    const uint32_t NW = nw_per_bin;
    P.nwave = NW;
    P.wdesc.clear();
    P.bin_of_cohort.assign(C, 0);
    int64_t bin = -1;        // open bin (-1: none)
    uint32_t wave = 0, lane = 0;
    // sub-wavefront class: free lanes and cohorts of the open bin's wavefronts
    std::vector<uint32_t> room(NW, 0u), ncoh(NW, 0u);
    uint32_t started = 0;    // wavefronts started in the open bin
    // multi-wavefront class: the bin before the open one, still open
    int64_t prev_bin = -1;
    uint32_t prev_used = 0;
    auto open_bin = [&]() {
        ++bin;
        wave = 0;
        lane = 0;
        started = 0;
        P.wdesc.resize((size_t)(bin + 1) * NW * WD_WORDS, 0u);
    };
    auto place = [&](uint32_t c) {
        const uint32_t b = off[c], k = off[c + 1] - off[c];
        if (k > 64u) {
            // The previous bin stays open beside the current one: a cohort
            // goes into the first of the two with nw free wavefronts left,
            // else into a new bin (which retires the previous one).  So a
            // cohort lands at most one bin before the one of any cohort
            // placed earlier; bins_of_range widens its range by one.
            const uint32_t nw = (k + 63u) / 64u;
            int64_t tb;
            uint32_t tw;
            if (prev_bin >= 0 && prev_used + nw <= NW) {
                tb = prev_bin;
                tw = prev_used;
                prev_used += nw;
            } else {
                if (bin < 0 || wave + nw > NW) {
                    prev_bin = bin;  // -1 before the class's first bin
                    prev_used = wave;
                    open_bin();
                }
                tb = bin;
                tw = wave;
                wave += nw;
            }
            for (uint32_t i = 0; i < nw; ++i) {
                uint32_t* d = &P.wdesc[((size_t)tb * NW + tw + i) * WD_WORDS];
                d[WD_S0] = b + 64u * i;
                d[WD_NACT] = (k - 64u * i) < 64u ? (k - 64u * i) : 64u;
                d[WD_CFIRST] = c;
                d[WD_NCOH] = 1;
                d[WD_BFIRST] = b;
                d[WD_KFIRST] = k;
                d[WD_FLAGS] = WF_MULTI | (i << 8) | (nw << 16) | (tw << 24);
            }
            P.bin_of_cohort[c] = (uint32_t)tb;
        } else {
            // first fit among the wavefronts of the open bin (so that the
            // bins of a cohort range stay together), then a new wavefront
            uint32_t w = NW;
            if (bin >= 0)
                for (uint32_t q = 0; q < started; ++q)
                    if (room[q] >= k && ncoh[q] < WD_MAXC) { w = q; break; }
            if (w == NW) {
                if (bin < 0 || started == NW) open_bin();
                w = started++;
                room[w] = 64u;
                ncoh[w] = 0u;
                uint32_t* d = &P.wdesc[((size_t)bin * NW + w) * WD_WORDS];
                d[WD_S0] = b;
                d[WD_NACT] = 0;
                d[WD_CFIRST] = c;
                d[WD_NCOH] = 0;
                d[WD_BFIRST] = b;
                d[WD_KFIRST] = k;
                d[WD_FLAGS] = 0;
            }
            uint32_t* d = &P.wdesc[((size_t)bin * NW + w) * WD_WORDS];
            d[WD_LIST + ncoh[w]] = c;
            d[WD_NCOH] = ++ncoh[w];
            d[WD_NACT] += k;
            room[w] -= k;
            P.bin_of_cohort[c] = (uint32_t)bin;
        }
    };
    for (uint32_t c = 0; c < C; ++c)
        if (off[c + 1] - off[c] <= 64u) place(c);
    P.n_bins_a = (uint32_t)(bin + 1);
    wave = NW;  // the multi-wavefront class starts in a fresh bin
    lane = 0;
    prev_bin = -1;
    for (uint32_t c = 0; c < C; ++c)
        if (off[c + 1] - off[c] > 64u) place(c);
    P.n_bins = (uint32_t)(bin + 1);

    // class lookups for cohort ranges
    P.first_a.assign(C + 1u, C);
    P.first_b.assign(C + 1u, C);
    for (int64_t c = (int64_t)C - 1; c >= 0; --c) {
        const bool small = off[c + 1] - off[c] <= 64u;
        P.first_a[c] = small ? (uint32_t)c : P.first_a[c + 1];
        P.first_b[c] = small ? P.first_b[c + 1] : (uint32_t)c;
    }
    P.last_a.assign(C, -1);
    P.last_b.assign(C, -1);
    for (uint32_t c = 0; c < C; ++c) {
        const bool small = off[c + 1] - off[c] <= 64u;
        P.last_a[c] = small ? (int32_t)c : (c ? P.last_a[c - 1] : -1);
        P.last_b[c] = small ? (c ? P.last_b[c - 1] : -1) : (int32_t)c;
    }

    // mark workgroups that contain a multi-wavefront cohort; count idle lanes
    uint32_t idle = 0;
    for (uint32_t bb = 0; bb < P.n_bins; ++bb) {
        bool any = false;
        for (uint32_t w = 0; w < NW; ++w) any |= (P.wdesc[((size_t)bb * NW + w) * WD_WORDS + WD_FLAGS] & WF_MULTI) != 0u;
        for (uint32_t w = 0; w < NW; ++w) {
            uint32_t* d = &P.wdesc[((size_t)bb * NW + w) * WD_WORDS];
            if (any) d[WD_FLAGS] |= WF_WGMULTI;
            idle += 64u - d[WD_NACT];
        }
    }
    P.idle_lanes = idle;
}

// Bins covering the cohorts [cb, ce) (cb < ce): a range of sub-wavefront
// bins and a range of multi-wavefront bins.
void bins_of_range(const Plan& P, uint32_t cb, uint32_t ce, uint32_t& a_lo, uint32_t& a_n,
                   uint32_t& b_lo, uint32_t& b_n) {
    a_lo = a_n = b_lo = b_n = 0;
    const uint32_t fa = P.first_a[cb];
    if (fa < ce) {
        const uint32_t la = (uint32_t)P.last_a[ce - 1];
        a_lo = P.bin_of_cohort[fa];
        a_n = P.bin_of_cohort[la] - a_lo + 1u;
    }
    const uint32_t fb = P.first_b[cb];
    if (fb < ce) {
        // a multi-wavefront cohort lies at most one bin before the bin of
        // any cohort placed earlier (build_plan), so the range's cohorts lie
        // within one bin of [bin(first), bin(last)]; cohorts of the extra
        // bins outside [cb, ce) are masked off in the kernels
        const uint32_t lb = (uint32_t)P.last_b[ce - 1];
        const uint32_t lo = P.bin_of_cohort[fb] > P.n_bins_a ? P.bin_of_cohort[fb] - 1u : P.n_bins_a;
        const uint32_t hi = P.bin_of_cohort[lb] + 1u < P.n_bins ? P.bin_of_cohort[lb] + 1u : P.n_bins - 1u;
        b_lo = lo;
        b_n = hi - lo + 1u;
    }
}

}  // namespace rc_plan

using namespace rc_plan;

extern "C" {

const char* rc_status_string(int status) {
    switch (status) {
        case RC_OK: return "RC_OK";
        case RC_E_INVALID: return "RC_E_INVALID";
        case RC_E_NOMEM: return "RC_E_NOMEM";
        case RC_E_DEVICE: return "RC_E_DEVICE";
        default: return "RC_E_UNKNOWN";
    }
}

int rc_plan_lanes(const rc_cohort_desc* desc, uint32_t lanes_per_workgroup, uint32_t* lane_session,
                  uint32_t* lane_cohort_out, uint32_t capacity, uint32_t* n_lanes) {
    if (!n_lanes) return RC_E_INVALID;
    const int v = validate_desc(desc);
    if (v != RC_OK) return v;
    if (lanes_per_workgroup != 256u && lanes_per_workgroup != 512u) return RC_E_INVALID;
    Plan P;
    build_plan(desc->cohort_offsets, desc->n_cohorts, lanes_per_workgroup / 64u, P);
    const uint32_t total = P.n_bins * lanes_per_workgroup;
    *n_lanes = total;
    if (!lane_session || !lane_cohort_out) return RC_OK;
    if (capacity < total) return RC_E_INVALID;
    const uint32_t* off = desc->cohort_offsets;
    for (uint32_t wv = 0; wv < P.n_bins * P.nwave; ++wv) {
        const uint32_t* d = &P.wdesc[(size_t)wv * WD_WORDS];
        for (uint32_t lane = 0; lane < 64u; ++lane) {
            // the per-lane derivation of lane_cohort() in the kernels
            uint32_t s = d[WD_S0] + lane;
            uint32_t c = d[WD_CFIRST];
            if (d[WD_NCOH] > 1u) {
                uint32_t at = 0u;
                for (uint32_t q = 0; q < d[WD_NCOH]; ++q) {
                    const uint32_t cq = d[WD_LIST + q];
                    if (lane >= at) {
                        c = cq;
                        s = off[cq] + (lane - at);
                    }
                    at += off[cq + 1u] - off[cq];
                }
            }
            const bool act = lane < d[WD_NACT];
            lane_session[wv * 64u + lane] = act ? s : 0xFFFFFFFFu;
            lane_cohort_out[wv * 64u + lane] = act ? c : 0xFFFFFFFFu;
        }
    }
    return RC_OK;
}

}  // extern "C"
