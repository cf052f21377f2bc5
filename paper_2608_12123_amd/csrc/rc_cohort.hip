// rc_cohort.hip -- batched ready-cohort control transition for AMD Instinct
// MI355X (gfx950): hand-written HIP kernels and the C ABI of rc_cohort.h.
//
// Kernels
//   rc_chain_kernel   device-resident chain (Section 7 "Device resident"):
//                     one launch runs T chained steps; state lives in VGPRs,
//                     decisions never leave the chip.
//   rc_decide_kernel  host-round-trip step, part 1 (Section 7 "Host round
//                     trip"): decide + compact, publish a 4-byte word.
//   rc_body_kernel    host-round-trip step, part 2: one route body over the
//                     compacted list the host selected.
//
// Data layout (HBM, structure of arrays, leading dimension ld): state
// [W][ld], outcome [ld], effects [T][ld] x {sid, tool} and [T][4][ld]
// payload, n_taken [T][C].  A wavefront's 64 lanes touch 64 consecutive
// sessions of one word row, so every state access is a fully coalesced
// 256-byte row segment.
//
// Launch plan (built on the host at create time).  Cohorts are packed in
// order into workgroups ("bins") of 256 or 512 lanes.  A cohort of at most
// 64 sessions never straddles a wavefront; a larger cohort starts on a
// wavefront boundary and spans whole wavefronts; no cohort straddles a
// workgroup.  Per wavefront the plan stores a 32-byte descriptor read with
// scalar loads.  The compaction (stable partition, taken first) is a
// wavefront ballot + mbcnt rank; a cohort spanning several wavefronts adds an
// LDS exchange of per-wavefront popcounts behind one workgroup barrier per
// step (double-buffered, so one barrier suffices).
//
// Per-word update, branch-free.  With d the decision, r the route:
//   sh = d ? 0 : (31 - r) mod 32      rotl by (r+1) mod 32 == rotr by sh
//   M  = d ? table[r][w mod 16]*(w+1) : 0     (row R of the LDS table is 0)
//   oo = d ? 0 : o
//   S' = (rotr(S, sh) ^ M) + oo       one v_alignbit_b32 + one v_xad_u32
// For w >= 16 the mask is the one of w - 16 plus table[r][w mod 16] << 4
// (exact modulo 2^32), one v_lshl_add_u32 per word instead of a multiply.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <new>
#include <vector>

#include "rc_cohort.h"

namespace {

// ---------------------------------------------------------------------------
// Device side
// ---------------------------------------------------------------------------

// MurmurHash3's 32-bit finalizer.
__device__ __forceinline__ uint32_t dev_fmix32(uint32_t h) {
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

__device__ __forceinline__ uint32_t rotr32(uint32_t x, uint32_t s) {
    return __builtin_amdgcn_alignbit(x, x, s);  // uses s mod 32
}

__device__ __forceinline__ uint32_t lane_rank(uint64_t m) {
    // number of set bits of m below this lane
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint32_t uni(uint32_t v) {
    return __builtin_amdgcn_readfirstlane(v);
}

// Wavefront descriptor of the launch plan (8 x u32).
enum : uint32_t {
    WD_S0 = 0,        // session of lane 0
    WD_NACT = 1,      // lanes [0, n_act) hold sessions s0 .. s0 + n_act - 1
    WD_CFIRST = 2,    // cohort of lane 0
    WD_NCOH = 3,      // cohorts present in this wavefront
    WD_BFIRST = 4,    // first session of cohort c_first
    WD_KFIRST = 5,    // size of cohort c_first
    WD_FLAGS = 6,
    WD_WORDS = 8
};
enum : uint32_t {
    WF_MULTI = 1u,    // this wavefront is part of a cohort of > 64 sessions
    WF_WGMULTI = 2u,  // some wavefront of the workgroup is (uniform per WG)
    // bits 8..15: index of this wavefront inside its cohort
    // bits 16..23: wavefronts of the cohort
    // bits 24..31: first wavefront (inside the workgroup) of the cohort
};

struct RouteArgs {
    uint32_t mode;      // RC_ROUTE_MOD / RC_ROUTE_CDF
    uint32_t n_routes;  // R
    uint32_t pow2_mask; // R - 1 when R is a power of two, else 0
    uint32_t is_pow2;
    uint32_t cdf_n;     // R - 1 thresholds
    uint32_t cdf_top;   // largest power of two <= cdf_n (0 if none)
};

// Route key (MOD: o mod R; CDF: number of thresholds <= o, found by a
// fixed-trip binary search over the LDS copy of the thresholds).
__device__ __forceinline__ uint32_t route_of(uint32_t o, const RouteArgs& ra,
                                             const uint32_t* cdf) {
    if (ra.mode == RC_ROUTE_MOD)
        return ra.is_pow2 ? (o & ra.pow2_mask) : (o % ra.n_routes);
    uint32_t pos = 0;
    for (uint32_t stp = ra.cdf_top; stp != 0u; stp >>= 1) {
        const uint32_t i = pos + stp;
        const uint32_t v = cdf[(i <= ra.cdf_n ? i : ra.cdf_n) - 1u];
        pos = (i <= ra.cdf_n && v <= o) ? i : pos;
    }
    return pos;
}

struct ChainArgs {
    uint32_t* state;
    uint32_t* outcome;
    uint32_t* eff_sid;
    uint32_t* eff_tool;
    uint32_t* eff_payload;
    uint32_t* n_taken;
    const uint32_t* tab;      // (R+1) x 16 swizzled rows, row R all zero
    const uint32_t* tools;    // [R] (table[r][0] & 7) | (table[r][1] & 7) << 8
    const uint32_t* cdf;      // [R-1]
    const uint32_t* offsets;  // [C+1]
    const uint32_t* wdesc;    // [bins][waves][WD_WORDS]
    RouteArgs ra;
    uint32_t ld, n_words, n_cohorts, thr, step0, n_steps;
    uint32_t cohort_begin, cohort_end, bin_lo, bin_hi;
    uint32_t lds_tools_off, lds_cdf_off, lds_cnt_off;  // in words
};

// Per-lane view of the plan for one bin.
struct LaneCohort {
    uint32_t s;       // session
    uint32_t c;       // cohort
    uint32_t b;       // first session of the cohort
    uint32_t k;       // cohort size
    uint64_t seg;     // lanes of the cohort inside this wavefront (sub-wave)
    uint32_t flags;
    bool active;
};

__device__ __forceinline__ LaneCohort lane_cohort(const uint32_t* __restrict__ wd,
                                                  const uint32_t* __restrict__ offsets,
                                                  uint32_t lane, uint32_t cb, uint32_t ce) {
    LaneCohort L;
    const uint32_t s0 = uni(wd[WD_S0]);
    const uint32_t n_act = uni(wd[WD_NACT]);
    const uint32_t c_first = uni(wd[WD_CFIRST]);
    const uint32_t n_coh = uni(wd[WD_NCOH]);
    uint32_t b = uni(wd[WD_BFIRST]);
    uint32_t k = uni(wd[WD_KFIRST]);
    L.flags = uni(wd[WD_FLAGS]);
    L.s = s0 + lane;
    L.c = c_first;
    if (n_coh > 1u) {
        // several sub-wavefront cohorts: find this lane's one
        for (uint32_t q = 1; q < n_coh; ++q) {
            const uint32_t bq = offsets[c_first + q];  // uniform address
            L.c = (bq <= L.s) ? c_first + q : L.c;
        }
        b = offsets[L.c];
        k = offsets[L.c + 1u] - b;
    }
    L.b = b;
    L.k = k;
    L.active = lane < n_act && L.c >= cb && L.c < ce;
    L.seg = 0;
    if (!(L.flags & WF_MULTI)) {
        uint32_t lo = b - s0;
        uint32_t hi = lo + k;
        lo = lo < 64u ? lo : 64u;
        hi = hi < 64u ? hi : 64u;
        const uint64_t below_hi = hi >= 64u ? ~0ull : ((1ull << hi) - 1ull);
        const uint64_t below_lo = lo >= 64u ? ~0ull : ((1ull << lo) - 1ull);
        L.seg = below_hi & ~below_lo;
    }
    return L;
}

// Stable-partition slot of this lane at one step.  Returns the slot; n1 gets
// the cohort's taken count.  `par` toggles once per workgroup barrier.
template <int NWAVE>
__device__ __forceinline__ uint32_t compact_slot(const LaneCohort& L, bool dk, uint32_t lane,
                                                 uint32_t wv, uint32_t* cnt_lds,
                                                 uint32_t& par, uint32_t& n1) {
    const uint64_t bal = __ballot(dk);
    uint32_t rank_t;
    if (!(L.flags & WF_MULTI)) {
        const uint64_t bs = bal & L.seg;
        n1 = (uint32_t)__popcll(bs);
        rank_t = lane_rank(bs);
    } else {
        n1 = 0;
        rank_t = 0;
    }
    if (L.flags & WF_WGMULTI) {
        uint32_t* cnt = cnt_lds + par * NWAVE;
        if ((L.flags & WF_MULTI) && lane == 0u)
            cnt[wv] = (uint32_t)__popcll(bal);
        __syncthreads();
        if (L.flags & WF_MULTI) {
            const uint32_t wi = (L.flags >> 8) & 0xFFu;
            const uint32_t nw = (L.flags >> 16) & 0xFFu;
            const uint32_t wf = L.flags >> 24;
            uint32_t before = 0, total = 0;
            for (uint32_t i = 0; i < nw; ++i) {
                const uint32_t ci = cnt[wf + i];
                total += ci;
                before += (i < wi) ? ci : 0u;
            }
            n1 = total;
            rank_t = before + lane_rank(bal);
        }
        par ^= 1u;
    }
    const uint32_t in_c = L.s - L.b;
    return L.b + (dk ? rank_t : n1 + (in_c - rank_t));
}

// Load one table row (16 words, 4 swizzled 16-byte blocks) from LDS.
__device__ __forceinline__ void load_row(const uint32_t* lds_tab, uint32_t row, uint32_t (&tw)[16]) {
    const uint4* r4 = reinterpret_cast<const uint4*>(lds_tab) + row * 4u;
#pragma unroll
    for (uint32_t q = 0; q < 4; ++q) {
        const uint4 v = r4[(q + row) & 3u];
        tw[4 * q + 0] = v.x;
        tw[4 * q + 1] = v.y;
        tw[4 * q + 2] = v.z;
        tw[4 * q + 3] = v.w;
    }
}

template <int NWAVE>
__device__ __forceinline__ void stage_tables(uint32_t* lds, const ChainArgs& a, uint32_t tid) {
    constexpr uint32_t WG = NWAVE * 64;
    const uint32_t n4 = (a.ra.n_routes + 1u) * 4u;  // uint4 per table
    const uint4* src = reinterpret_cast<const uint4*>(a.tab);
    uint4* dst = reinterpret_cast<uint4*>(lds);
    for (uint32_t i = tid; i < n4; i += WG) dst[i] = src[i];
    for (uint32_t i = tid; i < a.ra.n_routes; i += WG) lds[a.lds_tools_off + i] = a.tools[i];
    if (a.ra.mode == RC_ROUTE_CDF)
        for (uint32_t i = tid; i < a.ra.cdf_n; i += WG) lds[a.lds_cdf_off + i] = a.cdf[i];
}

// Device-resident chain: T steps per bin without leaving the kernel.
template <int WMAX, bool EXACT, int NWAVE>
__global__ __launch_bounds__(NWAVE * 64) void rc_chain_kernel(ChainArgs a) {
    extern __shared__ uint4 lds4[];
    uint32_t* lds = reinterpret_cast<uint32_t*>(lds4);
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wv = tid >> 6;
    const uint32_t W = a.n_words;
    const size_t ld = a.ld;

    stage_tables<NWAVE>(lds, a, tid);
    __syncthreads();
    const uint32_t* lds_tools = lds + a.lds_tools_off;
    const uint32_t* lds_cdf = lds + a.lds_cdf_off;
    uint32_t* lds_cnt = lds + a.lds_cnt_off;
    uint32_t par = 0;

    for (uint32_t bin = a.bin_lo + blockIdx.x; bin < a.bin_hi; bin += gridDim.x) {
        const LaneCohort L = lane_cohort(a.wdesc + ((size_t)bin * NWAVE + wv) * WD_WORDS,
                                         a.offsets, lane, a.cohort_begin, a.cohort_end);
        uint32_t S[WMAX];
        uint32_t o = 0;
#pragma unroll
        for (int w = 0; w < WMAX; ++w) S[w] = 0;
        if (L.active) {
#pragma unroll
            for (int w = 0; w < WMAX; ++w)
                if (EXACT || (uint32_t)w < W) S[w] = a.state[(size_t)w * ld + L.s];
            o = a.outcome[L.s];
        }

        for (uint32_t t = 0; t < a.n_steps; ++t) {
            const uint32_t step = a.step0 + t;
            const uint32_t r = route_of(o, a.ra, lds_cdf);
            const uint32_t h = dev_fmix32(S[0] ^ o ^ step);
            const bool dk = L.active && ((h & 0xFFFFu) < a.thr);
            uint32_t n1;
            const uint32_t slot = compact_slot<NWAVE>(L, dk, lane, wv, lds_cnt, par, n1);

            const uint32_t row = dk ? r : a.ra.n_routes;
            const uint32_t sh = dk ? 0u : ((31u - r) & 31u);
            const uint32_t oo = dk ? 0u : o;
            uint32_t tw[16];
            load_row(lds, row, tw);
            uint32_t M[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) M[j] = tw[j] * (uint32_t)(j + 1);
#pragma unroll
            for (int w = 0; w < WMAX; ++w) {
                const int j = w & 15;
                if (w >= 16) M[j] += tw[j] << 4;
                if (EXACT || (uint32_t)w < W) S[w] = (rotr32(S[w], sh) ^ M[j]) + oo;
            }
            const uint32_t tool = (lds_tools[r] >> (dk ? 8u : 0u)) & 7u;

            // slot - b < k always holds; the test keeps a compaction defect
            // from ever turning into a write outside the cohort's slots
            if (L.active && slot - L.b < L.k) {
                const size_t e = (size_t)t * ld + slot;
                a.eff_sid[e] = L.s;
                a.eff_tool[e] = tool;
#pragma unroll
                for (int q = 0; q < 4; ++q) a.eff_payload[((size_t)t * 4 + q) * ld + slot] = S[q];
                if (L.s == L.b) a.n_taken[(size_t)t * a.n_cohorts + L.c] = n1;
            }
            o = dev_fmix32(S[0]);
        }

        if (L.active) {
#pragma unroll
            for (int w = 0; w < WMAX; ++w)
                if (EXACT || (uint32_t)w < W) a.state[(size_t)w * ld + L.s] = S[w];
            a.outcome[L.s] = o;
        }
    }
}

// Host round trip, part 1: decide and compact one step.  Writes n_taken,
// appends (sid, slot) to the taken or not-taken list, and counts both
// populations in ctr[parity][0..1] (ctr[parity][0] is the 4-byte word the
// host reads).  Block 0 clears the other parity's counters for the next step.
struct DecideArgs {
    const uint32_t* state;
    const uint32_t* outcome;
    uint32_t* n_taken;
    uint2* list_taken;
    uint2* list_not;
    uint32_t* ctr;            // [2][2]
    const uint32_t* offsets;
    const uint32_t* wdesc;
    uint32_t thr, step, t_index, n_cohorts, n_sessions;
    uint32_t cohort_begin, cohort_end, bin_lo, bin_hi, parity;
};

template <int NWAVE>
__global__ __launch_bounds__(NWAVE * 64) void rc_decide_kernel(DecideArgs a) {
    __shared__ uint32_t cnt_lds[2 * NWAVE];
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wv = tid >> 6;
    uint32_t par = 0;
    if (blockIdx.x == 0 && tid == 0) {
        a.ctr[(a.parity ^ 1u) * 2u + 0u] = 0u;
        a.ctr[(a.parity ^ 1u) * 2u + 1u] = 0u;
    }
    for (uint32_t bin = a.bin_lo + blockIdx.x; bin < a.bin_hi; bin += gridDim.x) {
        const LaneCohort L = lane_cohort(a.wdesc + ((size_t)bin * NWAVE + wv) * WD_WORDS,
                                         a.offsets, lane, a.cohort_begin, a.cohort_end);
        uint32_t s0w = 0, o = 0;
        if (L.active) {
            s0w = a.state[L.s];
            o = a.outcome[L.s];
        }
        const bool dk = L.active && ((dev_fmix32(s0w ^ o ^ a.step) & 0xFFFFu) < a.thr);
        uint32_t n1;
        const uint32_t slot = compact_slot<NWAVE>(L, dk, lane, wv, cnt_lds, par, n1);
        if (L.active && L.s == L.b) a.n_taken[(size_t)a.t_index * a.n_cohorts + L.c] = n1;

        const uint64_t bt = __ballot(dk);
        const uint64_t bn = __ballot(L.active && !dk);
        uint32_t base_t = 0, base_n = 0;
        if (lane == 0u) {
            if (bt) base_t = atomicAdd(&a.ctr[a.parity * 2u + 0u], (uint32_t)__popcll(bt));
            if (bn) base_n = atomicAdd(&a.ctr[a.parity * 2u + 1u], (uint32_t)__popcll(bn));
        }
        base_t = uni(base_t);
        base_n = uni(base_n);
        const uint32_t at = dk ? base_t + lane_rank(bt) : base_n + lane_rank(bn);
        if (L.active && at < a.n_sessions && slot - L.b < L.k)
            (dk ? a.list_taken : a.list_not)[at] = make_uint2(L.s, slot);
    }
}

// Host round trip, part 2: the route body the host selected, over its list.
struct BodyArgs {
    uint32_t* state;
    uint32_t* outcome;
    uint32_t* eff_sid;
    uint32_t* eff_tool;
    uint32_t* eff_payload;
    const uint2* list;
    const uint32_t* tab;
    const uint32_t* tools;
    const uint32_t* cdf;
    RouteArgs ra;
    uint32_t ld, n_words, count, t_index, n_sessions;
};

template <int WMAX, bool EXACT, bool TAKEN>
__global__ __launch_bounds__(256) void rc_body_kernel(BodyArgs a) {
    __shared__ uint32_t cdf_lds[RC_MAX_ROUTES];
    const uint32_t tid = threadIdx.x;
    if (a.ra.mode == RC_ROUTE_CDF) {
        for (uint32_t i = tid; i < a.ra.cdf_n; i += 256u) cdf_lds[i] = a.cdf[i];
        __syncthreads();
    }
    const uint32_t i = blockIdx.x * 256u + tid;
    if (i >= a.count) return;
    const uint32_t W = a.n_words;
    const size_t ld = a.ld;
    const uint2 e = a.list[i];
    const uint32_t s = e.x, slot = e.y;
    if (s >= a.n_sessions || slot >= a.n_sessions) return;  // never taken by valid lists
    const uint32_t o = a.outcome[s];
    const uint32_t r = route_of(o, a.ra, cdf_lds);
    uint32_t S[WMAX];
#pragma unroll
    for (int w = 0; w < WMAX; ++w)
        S[w] = (EXACT || (uint32_t)w < W) ? a.state[(size_t)w * ld + s] : 0u;
    if (TAKEN) {
        uint32_t tw[16];
        const uint4* r4 = reinterpret_cast<const uint4*>(a.tab) + r * 4u;
#pragma unroll
        for (uint32_t q = 0; q < 4; ++q) {
            const uint4 v = r4[(q + r) & 3u];
            tw[4 * q + 0] = v.x;
            tw[4 * q + 1] = v.y;
            tw[4 * q + 2] = v.z;
            tw[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int w = 0; w < WMAX; ++w) S[w] ^= tw[w & 15] * (uint32_t)(w + 1);
    } else {
        const uint32_t sh = (31u - r) & 31u;
#pragma unroll
        for (int w = 0; w < WMAX; ++w) S[w] = rotr32(S[w], sh) + o;
    }
#pragma unroll
    for (int w = 0; w < WMAX; ++w)
        if (EXACT || (uint32_t)w < W) a.state[(size_t)w * ld + s] = S[w];
    const size_t eo = (size_t)a.t_index * ld + slot;
    a.eff_sid[eo] = s;
    a.eff_tool[eo] = (a.tools[r] >> (TAKEN ? 8u : 0u)) & 7u;
#pragma unroll
    for (int q = 0; q < 4; ++q) a.eff_payload[((size_t)a.t_index * 4 + q) * ld + slot] = S[q];
    a.outcome[s] = dev_fmix32(S[0]);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

typedef void (*ChainFn)(ChainArgs);
typedef void (*DecideFn)(DecideArgs);
typedef void (*BodyFn)(BodyArgs);

template <int WMAX, bool EXACT>
ChainFn chain_fn(uint32_t nwave) {
    return nwave == 8 ? rc_chain_kernel<WMAX, EXACT, 8> : rc_chain_kernel<WMAX, EXACT, 4>;
}

ChainFn pick_chain(uint32_t wmax, bool exact, uint32_t nwave) {
    switch (wmax) {
        case 4: return exact ? chain_fn<4, true>(nwave) : chain_fn<4, false>(nwave);
        case 8: return exact ? chain_fn<8, true>(nwave) : chain_fn<8, false>(nwave);
        case 16: return exact ? chain_fn<16, true>(nwave) : chain_fn<16, false>(nwave);
        case 32: return exact ? chain_fn<32, true>(nwave) : chain_fn<32, false>(nwave);
        default: return exact ? chain_fn<64, true>(nwave) : chain_fn<64, false>(nwave);
    }
}

template <int WMAX, bool EXACT>
BodyFn body_fn(bool taken) {
    return taken ? rc_body_kernel<WMAX, EXACT, true> : rc_body_kernel<WMAX, EXACT, false>;
}

BodyFn pick_body(uint32_t wmax, bool exact, bool taken) {
    switch (wmax) {
        case 4: return exact ? body_fn<4, true>(taken) : body_fn<4, false>(taken);
        case 8: return exact ? body_fn<8, true>(taken) : body_fn<8, false>(taken);
        case 16: return exact ? body_fn<16, true>(taken) : body_fn<16, false>(taken);
        case 32: return exact ? body_fn<32, true>(taken) : body_fn<32, false>(taken);
        default: return exact ? body_fn<64, true>(taken) : body_fn<64, false>(taken);
    }
}

DecideFn pick_decide(uint32_t nwave) {
    return nwave == 8 ? rc_decide_kernel<8> : rc_decide_kernel<4>;
}

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) { prev = -1; return; }
        ok = (prev == dev) || (hipSetDevice(dev) == hipSuccess);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

uint32_t next_pow2_words(uint32_t w) {
    uint32_t p = 4;
    while (p < w) p <<= 1;
    return p;
}

}  // namespace

struct rc_cohort {
    int device = -1;
    uint32_t N = 0, W = 0, R = 0, C = 0, thr = 0;
    RouteArgs ra{};
    uint32_t wmax = 4;
    bool exact = true;
    uint32_t nwave = 4;
    uint32_t n_bins = 0;
    uint32_t idle_lanes = 0;
    uint32_t max_grid = 1;
    size_t chain_lds_bytes = 0;
    uint32_t lds_tools_off = 0, lds_cdf_off = 0, lds_cnt_off = 0;
    std::vector<uint32_t> offsets;        // host copy [C+1]
    std::vector<uint32_t> bin_of_cohort;  // [C]
    uint32_t* d_offsets = nullptr;
    uint32_t* d_tab = nullptr;
    uint32_t* d_tools = nullptr;
    uint32_t* d_cdf = nullptr;
    uint32_t* d_wdesc = nullptr;
    uint2* d_list_taken = nullptr;
    uint2* d_list_not = nullptr;
    uint32_t* d_ctr = nullptr;
    uint32_t* h_word = nullptr;  // pinned
    uint32_t parity = 0;
    bool ctr_dirty = false;
    uint32_t last_launches = 0, last_d2h = 0;
};

namespace {

void free_handle(rc_cohort* h) {
    if (!h) return;
    if (h->device >= 0) {
        DeviceGuard g(h->device);
        (void)hipFree(h->d_offsets);
        (void)hipFree(h->d_tab);
        (void)hipFree(h->d_tools);
        (void)hipFree(h->d_cdf);
        (void)hipFree(h->d_wdesc);
        (void)hipFree(h->d_list_taken);
        (void)hipFree(h->d_list_not);
        (void)hipFree(h->d_ctr);
        if (h->h_word) (void)hipHostFree(h->h_word);
    }
    delete h;
}

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

// Pack cohorts into workgroups of nwave wavefronts (see the file comment).
void build_plan(rc_cohort* h, std::vector<uint32_t>& wdesc) {
    const uint32_t NW = h->nwave;
    const std::vector<uint32_t>& off = h->offsets;
    wdesc.clear();
    h->bin_of_cohort.assign(h->C, 0);
    uint32_t bin = 0, wave = 0, lane = 0;  // next free position
    auto ensure_bin = [&](uint32_t b) {
        if (wdesc.size() < (size_t)(b + 1) * NW * WD_WORDS) wdesc.resize((size_t)(b + 1) * NW * WD_WORDS, 0u);
    };
    ensure_bin(0);
    for (uint32_t c = 0; c < h->C; ++c) {
        const uint32_t b = off[c], k = off[c + 1] - off[c];
        if (k > 64u) {
            const uint32_t nw = (k + 63u) / 64u;
            if (lane > 0u) { ++wave; lane = 0; }
            if (wave + nw > NW) { ++bin; wave = 0; lane = 0; }
            ensure_bin(bin);
            for (uint32_t i = 0; i < nw; ++i) {
                uint32_t* d = &wdesc[((size_t)bin * NW + wave + i) * WD_WORDS];
                d[WD_S0] = b + 64u * i;
                d[WD_NACT] = (k - 64u * i) < 64u ? (k - 64u * i) : 64u;
                d[WD_CFIRST] = c;
                d[WD_NCOH] = 1;
                d[WD_BFIRST] = b;
                d[WD_KFIRST] = k;
                d[WD_FLAGS] = WF_MULTI | (i << 8) | (nw << 16) | (wave << 24);
            }
            h->bin_of_cohort[c] = bin;
            wave += nw;
            lane = 0;
        } else {
            if (lane + k > 64u) { ++wave; lane = 0; }
            if (wave >= NW) { ++bin; wave = 0; lane = 0; }
            ensure_bin(bin);
            uint32_t* d = &wdesc[((size_t)bin * NW + wave) * WD_WORDS];
            if (lane == 0u) {
                d[WD_S0] = b;
                d[WD_NACT] = 0;
                d[WD_CFIRST] = c;
                d[WD_NCOH] = 0;
                d[WD_BFIRST] = b;
                d[WD_KFIRST] = k;
                d[WD_FLAGS] = 0;
            }
            d[WD_NACT] += k;
            d[WD_NCOH] += 1;
            h->bin_of_cohort[c] = bin;
            lane += k;
        }
    }
    h->n_bins = (uint32_t)(wdesc.size() / ((size_t)NW * WD_WORDS));
    // mark workgroups that contain a multi-wavefront cohort; count idle lanes
    uint32_t idle = 0;
    for (uint32_t bb = 0; bb < h->n_bins; ++bb) {
        bool any = false;
        for (uint32_t w = 0; w < NW; ++w) any |= (wdesc[((size_t)bb * NW + w) * WD_WORDS + WD_FLAGS] & WF_MULTI) != 0u;
        for (uint32_t w = 0; w < NW; ++w) {
            uint32_t* d = &wdesc[((size_t)bb * NW + w) * WD_WORDS];
            if (any) d[WD_FLAGS] |= WF_WGMULTI;
            idle += 64u - d[WD_NACT];
        }
    }
    h->idle_lanes = idle;
}

template <typename T>
int dev_upload(T** dst, const void* src, size_t bytes) {
    if (hipMalloc((void**)dst, bytes < 16 ? 16 : bytes) != hipSuccess) return RC_E_NOMEM;
    if (bytes && hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice) != hipSuccess) return RC_E_DEVICE;
    return RC_OK;
}

// Is [p, p + bytes) inside one HIP allocation of device `dev`?
bool device_extent_ok(const void* p, size_t bytes, int dev) {
    if (!p) return false;
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) { (void)hipGetLastError(); return false; }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) return false;
    if (attr.device != dev) return false;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) != hipSuccess) { (void)hipGetLastError(); return false; }
    const uintptr_t b = (uintptr_t)base, q = (uintptr_t)p;
    return q >= b && q - b <= size && bytes <= size - (q - b);
}

int validate_buffers(const rc_cohort* h, const rc_buffers* b, uint32_t T) {
    if (!b) return RC_E_INVALID;
    if (b->ld < h->N) return RC_E_INVALID;
    const uint64_t ld = b->ld;
    struct Ext { const void* p; uint64_t bytes; } ext[6] = {
        {b->state, 4ull * h->W * ld},
        {b->outcome, 4ull * ld},
        {b->eff_sid, 4ull * T * ld},
        {b->eff_tool, 4ull * T * ld},
        {b->eff_payload, 16ull * T * ld},
        {b->n_taken, 4ull * T * h->C},
    };
    for (int i = 0; i < 6; ++i) {
        if (!ext[i].p) return RC_E_INVALID;
        if (ext[i].bytes >= (1ull << 46)) return RC_E_INVALID;
    }
    for (int i = 0; i < 6; ++i)
        for (int j = i + 1; j < 6; ++j) {
            const uintptr_t a0 = (uintptr_t)ext[i].p, a1 = a0 + ext[i].bytes;
            const uintptr_t b0 = (uintptr_t)ext[j].p, b1 = b0 + ext[j].bytes;
            if (a0 < b1 && b0 < a1) return RC_E_INVALID;
        }
    for (int i = 0; i < 6; ++i)
        if (!device_extent_ok(ext[i].p, ext[i].bytes, h->device)) return RC_E_INVALID;
    return RC_OK;
}

ChainArgs chain_args(const rc_cohort* h, const rc_buffers* b) {
    ChainArgs a;
    a.state = b->state;
    a.outcome = b->outcome;
    a.eff_sid = b->eff_sid;
    a.eff_tool = b->eff_tool;
    a.eff_payload = b->eff_payload;
    a.n_taken = b->n_taken;
    a.tab = h->d_tab;
    a.tools = h->d_tools;
    a.cdf = h->d_cdf;
    a.offsets = h->d_offsets;
    a.wdesc = h->d_wdesc;
    a.ra = h->ra;
    a.ld = b->ld;
    a.n_words = h->W;
    a.n_cohorts = h->C;
    a.thr = h->thr;
    a.lds_tools_off = h->lds_tools_off;
    a.lds_cdf_off = h->lds_cdf_off;
    a.lds_cnt_off = h->lds_cnt_off;
    return a;
}

int launch_ok() {
    return hipGetLastError() == hipSuccess ? RC_OK : RC_E_DEVICE;
}

int run_resident(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t T,
                 uint32_t cb, uint32_t ce, hipStream_t stream) {
    ChainArgs a = chain_args(h, b);
    a.step0 = step0;
    a.n_steps = T;
    a.cohort_begin = cb;
    a.cohort_end = ce;
    a.bin_lo = h->bin_of_cohort[cb];
    a.bin_hi = h->bin_of_cohort[ce - 1] + 1u;
    const uint32_t bins = a.bin_hi - a.bin_lo;
    const uint32_t grid = bins < h->max_grid ? bins : h->max_grid;
    ChainFn fn = pick_chain(h->wmax, h->exact, h->nwave);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(h->nwave * 64), h->chain_lds_bytes, stream, a);
    if (launch_ok() != RC_OK) return RC_E_DEVICE;
    h->last_launches = 1;
    h->last_d2h = 0;
    return RC_OK;
}

int run_host_roundtrip(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t T,
                       uint32_t cb, uint32_t ce, hipStream_t stream) {
    uint32_t launches = 0, copies = 0;
    if (h->ctr_dirty) {
        if (hipMemsetAsync(h->d_ctr, 0, 4 * sizeof(uint32_t), stream) != hipSuccess) return RC_E_DEVICE;
        h->parity = 0;
        h->ctr_dirty = false;
    }
    const uint32_t bin_lo = h->bin_of_cohort[cb];
    const uint32_t bin_hi = h->bin_of_cohort[ce - 1] + 1u;
    const uint32_t bins = bin_hi - bin_lo;
    const uint32_t grid = bins < h->max_grid ? bins : h->max_grid;
    const uint32_t n_range = h->offsets[ce] - h->offsets[cb];
    DecideFn dfn = pick_decide(h->nwave);
    BodyFn taken_fn = pick_body(h->wmax, h->exact, true);
    BodyFn not_fn = pick_body(h->wmax, h->exact, false);
    for (uint32_t t = 0; t < T; ++t) {
        h->ctr_dirty = true;  // cleared again when the step completes
        DecideArgs d;
        d.state = b->state;
        d.outcome = b->outcome;
        d.n_taken = b->n_taken;
        d.list_taken = h->d_list_taken;
        d.list_not = h->d_list_not;
        d.ctr = h->d_ctr;
        d.offsets = h->d_offsets;
        d.wdesc = h->d_wdesc;
        d.thr = h->thr;
        d.step = step0 + t;
        d.t_index = t;
        d.n_cohorts = h->C;
        d.n_sessions = h->N;
        d.cohort_begin = cb;
        d.cohort_end = ce;
        d.bin_lo = bin_lo;
        d.bin_hi = bin_hi;
        d.parity = h->parity;
        hipLaunchKernelGGL(dfn, dim3(grid), dim3(h->nwave * 64), 0, stream, d);
        if (launch_ok() != RC_OK) return RC_E_DEVICE;
        ++launches;
        // the observation: 4 bytes to pinned host memory, then wait
        if (hipMemcpyAsync(h->h_word, h->d_ctr + h->parity * 2u, sizeof(uint32_t),
                           hipMemcpyDeviceToHost, stream) != hipSuccess) return RC_E_DEVICE;
        ++copies;
        if (hipStreamSynchronize(stream) != hipSuccess) return RC_E_DEVICE;
        const uint32_t n_taken_total = *h->h_word;
        if (n_taken_total > n_range) return RC_E_DEVICE;
        // the host branch: launch the selected route body (or both)
        BodyArgs ba;
        ba.state = b->state;
        ba.outcome = b->outcome;
        ba.eff_sid = b->eff_sid;
        ba.eff_tool = b->eff_tool;
        ba.eff_payload = b->eff_payload;
        ba.tab = h->d_tab;
        ba.tools = h->d_tools;
        ba.cdf = h->d_cdf;
        ba.ra = h->ra;
        ba.ld = b->ld;
        ba.n_words = h->W;
        ba.t_index = t;
        ba.n_sessions = h->N;
        if (n_taken_total > 0u) {
            ba.list = h->d_list_taken;
            ba.count = n_taken_total;
            hipLaunchKernelGGL(taken_fn, dim3((n_taken_total + 255u) / 256u), dim3(256), 0, stream, ba);
            if (launch_ok() != RC_OK) return RC_E_DEVICE;
            ++launches;
        }
        if (n_taken_total < n_range) {
            ba.list = h->d_list_not;
            ba.count = n_range - n_taken_total;
            hipLaunchKernelGGL(not_fn, dim3((ba.count + 255u) / 256u), dim3(256), 0, stream, ba);
            if (launch_ok() != RC_OK) return RC_E_DEVICE;
            ++launches;
        }
        h->parity ^= 1u;
        h->ctr_dirty = false;
    }
    h->last_launches = launches;
    h->last_d2h = copies;
    return RC_OK;
}

}  // namespace

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

int rc_cohort_create(const rc_cohort_desc* desc, int hip_device, rc_cohort** out) {
    if (!out) return RC_E_INVALID;
    const int v = validate_desc(desc);
    if (v != RC_OK) return v;

    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev <= 0) { (void)hipGetLastError(); return RC_E_DEVICE; }
    if (hip_device < 0 || hip_device >= n_dev) return RC_E_DEVICE;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, hip_device) != hipSuccess) return RC_E_DEVICE;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return RC_E_DEVICE;

    rc_cohort* h = new (std::nothrow) rc_cohort();
    if (!h) return RC_E_NOMEM;
    DeviceGuard guard(hip_device);
    if (!guard.ok) { delete h; return RC_E_DEVICE; }
    h->device = hip_device;
    h->N = desc->n_sessions;
    h->W = desc->n_words;
    h->R = desc->n_routes;
    h->C = desc->n_cohorts;
    h->thr = desc->decide_thr;
    h->wmax = next_pow2_words(h->W);
    h->exact = (h->wmax == h->W);
    h->ra.mode = desc->route_mode;
    h->ra.n_routes = h->R;
    h->ra.is_pow2 = (h->R & (h->R - 1u)) == 0u;
    h->ra.pow2_mask = h->ra.is_pow2 ? h->R - 1u : 0u;
    h->ra.cdf_n = (desc->route_mode == RC_ROUTE_CDF) ? h->R - 1u : 0u;
    h->ra.cdf_top = 0;
    while (h->ra.cdf_n && (h->ra.cdf_top << 1) <= h->ra.cdf_n && h->ra.cdf_top < (1u << 30))
        h->ra.cdf_top = h->ra.cdf_top ? h->ra.cdf_top << 1 : 1u;

    // LDS image: (R+1) x 16 table words, rows 64 B with the four 16-byte
    // blocks of row r rotated by r (bank spreading), row R all zero; then the
    // packed tool pairs, the CDF thresholds and the popcount exchange.
    const uint32_t R = h->R;
    std::vector<uint32_t> tab((size_t)(R + 1) * 16u, 0u), tools(R, 0u);
    for (uint32_t r = 0; r < R; ++r) {
        for (uint32_t j = 0; j < 16; ++j) {
            const uint32_t q = j >> 2, p = ((q + r) & 3u) * 4u + (j & 3u);
            tab[(size_t)r * 16u + p] = desc->table[(size_t)r * 16u + j];
        }
        tools[r] = (desc->table[(size_t)r * 16u + 0] & 7u) | ((desc->table[(size_t)r * 16u + 1] & 7u) << 8);
    }
    const uint32_t tab_words = (R + 1u) * 16u;
    h->lds_tools_off = tab_words;
    h->lds_cdf_off = h->lds_tools_off + ((R + 3u) & ~3u);
    h->lds_cnt_off = h->lds_cdf_off + ((h->ra.cdf_n + 3u) & ~3u);
    const size_t lds_words = h->lds_cnt_off + 2u * 8u;
    h->chain_lds_bytes = lds_words * 4u;
    h->nwave = h->chain_lds_bytes > 40u * 1024u ? 8u : 4u;

    h->offsets.assign(desc->cohort_offsets, desc->cohort_offsets + h->C + 1u);
    std::vector<uint32_t> wdesc;
    build_plan(h, wdesc);

    int rc = RC_OK;
    if (rc == RC_OK) rc = dev_upload(&h->d_offsets, h->offsets.data(), h->offsets.size() * 4u);
    if (rc == RC_OK) rc = dev_upload(&h->d_tab, tab.data(), tab.size() * 4u);
    if (rc == RC_OK) rc = dev_upload(&h->d_tools, tools.data(), tools.size() * 4u);
    if (rc == RC_OK) {
        if (h->ra.cdf_n) rc = dev_upload(&h->d_cdf, desc->route_cdf, (size_t)h->ra.cdf_n * 4u);
        else rc = dev_upload(&h->d_cdf, nullptr, 0);
    }
    if (rc == RC_OK) rc = dev_upload(&h->d_wdesc, wdesc.data(), wdesc.size() * 4u);
    if (rc == RC_OK && hipMalloc((void**)&h->d_list_taken, (size_t)h->N * sizeof(uint2)) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMalloc((void**)&h->d_list_not, (size_t)h->N * sizeof(uint2)) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMalloc((void**)&h->d_ctr, 4 * sizeof(uint32_t)) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMemset(h->d_ctr, 0, 4 * sizeof(uint32_t)) != hipSuccess) rc = RC_E_DEVICE;
    if (rc == RC_OK && hipHostMalloc((void**)&h->h_word, sizeof(uint32_t), hipHostMallocDefault) != hipSuccess) rc = RC_E_NOMEM;

    if (rc == RC_OK) {
        ChainFn fn = pick_chain(h->wmax, h->exact, h->nwave);
        if (hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)h->chain_lds_bytes) != hipSuccess) rc = RC_E_DEVICE;
        int per_cu = 0;
        if (rc == RC_OK && hipOccupancyMaxActiveBlocksPerMultiprocessor(
                               &per_cu, (const void*)fn, (int)(h->nwave * 64), h->chain_lds_bytes) != hipSuccess)
            rc = RC_E_DEVICE;
        if (rc == RC_OK) {
            if (per_cu < 1) per_cu = 1;
            h->max_grid = (uint32_t)per_cu * (uint32_t)prop.multiProcessorCount;
        }
    }
    if (rc != RC_OK) {
        (void)hipGetLastError();
        free_handle(h);
        return rc;
    }
    *out = h;
    return RC_OK;
}

int rc_cohort_run_chain(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t n_steps,
                        int mode, uint32_t cohort_begin, uint32_t cohort_end, void* hip_stream) {
    if (!h || !b) return RC_E_INVALID;
    if (mode != RC_MODE_RESIDENT && mode != RC_MODE_HOST_ROUNDTRIP) return RC_E_INVALID;
    if (cohort_begin > cohort_end || cohort_end > h->C) return RC_E_INVALID;
    DeviceGuard guard(h->device);
    if (!guard.ok) return RC_E_DEVICE;
    const int v = validate_buffers(h, b, n_steps);
    if (v != RC_OK) return v;
    h->last_launches = 0;
    h->last_d2h = 0;
    if (n_steps == 0u || cohort_begin == cohort_end) return RC_OK;
    hipStream_t stream = (hipStream_t)hip_stream;
    if (mode == RC_MODE_RESIDENT) return run_resident(h, b, step0, n_steps, cohort_begin, cohort_end, stream);
    return run_host_roundtrip(h, b, step0, n_steps, cohort_begin, cohort_end, stream);
}

int rc_cohort_step(rc_cohort* h, const rc_buffers* b, uint32_t step, uint32_t cohort_begin,
                   uint32_t cohort_end, void* hip_stream) {
    return rc_cohort_run_chain(h, b, step, 1u, RC_MODE_RESIDENT, cohort_begin, cohort_end, hip_stream);
}

int rc_cohort_destroy(rc_cohort* h) {
    free_handle(h);
    return RC_OK;
}

int rc_cohort_last_counts(const rc_cohort* h, uint32_t* launches, uint32_t* d2h_copies) {
    if (!h) return RC_E_INVALID;
    if (launches) *launches = h->last_launches;
    if (d2h_copies) *d2h_copies = h->last_d2h;
    return RC_OK;
}

int rc_cohort_plan_info(const rc_cohort* h, uint32_t* n_workgroups, uint32_t* lanes_per_workgroup,
                        uint32_t* idle_lanes) {
    if (!h) return RC_E_INVALID;
    if (n_workgroups) *n_workgroups = h->n_bins;
    if (lanes_per_workgroup) *lanes_per_workgroup = h->nwave * 64u;
    if (idle_lanes) *idle_lanes = h->idle_lanes;
    return RC_OK;
}

}  // extern "C"
