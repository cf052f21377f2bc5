// rc_plan.h -- launch plan of the ready-cohort chain kernels (internal,
// host side; not part of the C ABI).  Shared by the HIP library and its
// host-only part (rc_host.cpp), which also builds without any GPU toolchain.
#ifndef RC_PLAN_H
#define RC_PLAN_H

#include <stdint.h>

#include <vector>

#include "rc_cohort.h"

namespace rc_plan {

// Wavefront descriptor of the launch plan (16 x u32).
enum : uint32_t {
    WD_S0 = 0,        // session of lane 0
    WD_NACT = 1,      // lanes [0, n_act) are active
    WD_CFIRST = 2,    // cohort of lane 0
    WD_NCOH = 3,      // cohorts present in this wavefront
    WD_BFIRST = 4,    // first session of cohort c_first
    WD_KFIRST = 5,    // size of cohort c_first
    WD_FLAGS = 6,
    WD_LIST = 8,      // sub-wavefront cohorts, in lane order: cohort q takes the
                      // next k_q lanes, which hold its sessions in order
    WD_MAXC = 8,      // at most this many cohorts per wavefront
    WD_WORDS = 16
};
enum : uint32_t {
    WF_MULTI = 1u,    // this wavefront is part of a cohort of > 64 sessions
    WF_WGMULTI = 2u,  // some wavefront of the workgroup is (uniform per WG)
    // bits 8..15: index of this wavefront inside its cohort
    // bits 16..23: wavefronts of the cohort (at most 4)
    // bits 24..31: first wavefront (inside the workgroup) of the cohort
};

// The launch plan: per-wavefront descriptors plus the lookups that turn a
// cohort range into bin ranges.  Built on the host, without a device.
struct Plan {
    uint32_t nwave = 4;
    uint32_t n_bins = 0, n_bins_a = 0, idle_lanes = 0;
    std::vector<uint32_t> wdesc;             // [bins][nwave][WD_WORDS]
    std::vector<uint32_t> bin_of_cohort;     // [C]
    std::vector<uint32_t> first_a, first_b;  // [C+1]: first cohort >= c of the class (C if none)
    std::vector<int32_t> last_a, last_b;     // [C]: last cohort <= c of the class (-1 if none)
};

// RC_OK, or RC_E_INVALID for a descriptor outside the limits of rc_cohort.h.
int validate_desc(const rc_cohort_desc* d);

// Pack cohorts into bins of nw_per_bin wavefronts.
void build_plan(const uint32_t* off, uint32_t C, uint32_t nw_per_bin, Plan& P);

// Bins covering the cohorts [cb, ce) (cb < ce): a range of sub-wavefront
// bins and a range of multi-wavefront bins.
void bins_of_range(const Plan& P, uint32_t cb, uint32_t ce, uint32_t& a_lo, uint32_t& a_n,
                   uint32_t& b_lo, uint32_t& b_n);

}  // namespace rc_plan

#endif  // RC_PLAN_H
