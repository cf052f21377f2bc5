// rc_cohort.hip -- batched ready-cohort control transition for AMD Instinct
// MI355X (gfx950): hand-written HIP kernels and the C ABI of rc_cohort.h.
//
// Kernels
//   rc_prep_kernel    once per handle: builds the route-table image that every
//                     workgroup stages into LDS.
//   rc_chain_kernel   device-resident chain (Section 7 "Device resident"):
//                     one launch runs T chained steps; state lives in VGPRs,
//                     decisions never leave the chip.
//   rc_decide_kernel  host-round-trip step, part 1 (Section 7 "Host round
//                     trip"): decide + compact, publish a 4-byte word.
//   rc_body_kernel    host-round-trip step, part 2: one route body over the
//                     compacted list the host selected.
//
// Data layout (HBM, structure of arrays, leading dimension ld): state
// [W][ld], outcome [ld], effects [T][ld] for sid and tool, [T][ld][4] for the
// payload, n_taken [T][C].  A wavefront's lanes read the consecutive
// sessions of each of its cohorts from one word row (at most a few
// contiguous segments per row); an effect's payload is one 16-byte store.
//
// Launch plan (built on the host at create time).  Cohorts of at most 64
// sessions are packed, in order, into "sub-wavefront" bins that never need a
// workgroup barrier -- each into the first wavefront of the open bin with room
// for it, so a wavefront can hold several cohorts that are not neighbours --
// and larger cohorts go, in order, into "multi-wavefront" bins.  A bin is one
// workgroup of 4 or 8 wavefronts.  A cohort of at most 64 sessions never
// straddles a wavefront; a larger one starts on a wavefront boundary and spans
// whole wavefronts; no cohort straddles a bin.  Each wavefront has a 64-byte
// descriptor read with scalar loads.  The compaction
// (stable partition, taken first) is a wavefront ballot + mbcnt rank; a
// cohort spanning wavefronts adds an LDS exchange of per-wavefront popcounts
// behind one workgroup barrier per step.
//
// Route-table image in LDS.
//   full:  row r < R holds the W masks table[r][w mod 16] * (w + 1); row R is
//          zero.  No arithmetic is left for the masks.
//   table: (when the full image would not fit) row r holds table[r][0..15],
//          row R is zero; the masks are formed in registers with full-rate
//          shifts and adds: the mask of w + 16 is the mask of w plus
//          table[r][w mod 16] << 4 (exact modulo 2^32).
// Block q (16 bytes) of row r is stored at block q ^ (r mod blocks-per-row)
// to spread lanes reading different rows over the LDS banks.  After the rows
// come the tool pairs (full image), the route thresholds and, in CDF mode, a
// guide table: guide[b] is the route of outcome b * 2^(32-g), so the route
// of o lies in [guide[o >> (32-g)], guide[(o >> (32-g)) + 1]] and a short
// binary search of fixed trip count finishes it (the indexed-search guide
// table of Chen and Asau, 1974).
//
// Per-word update, branch-free.  With d the decision and r the route:
//   sh = d ? 0 : (31 - r) mod 32      rotl by (r+1) mod 32 == rotr by sh
//   M  = masks of row (d ? r : R)      (zero when not taken)
//   oo = d ? 0 : o
//   S' = (rotr(S, sh) ^ M) + oo       one v_alignbit_b32 + one v_xad_u32
//
// Step schedule.  The decision of step t + 1 needs only word 0 after step
// t, so it is made right after words 0..3 are updated; its popcount is
// published and the workgroup barrier is passed there, the next mask row is
// prefetched, and only then are the remaining words updated -- so the
// barrier, the count exchange and the LDS latency overlap the bulk update.
// The effects of step t are stored at the end of step t.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <type_traits>
#include <vector>

#include "rc_cohort.h"
#include "rc_plan.h"



namespace {

using namespace rc_plan;

// ---------------------------------------------------------------------------
// Device helpers
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

// Hide a value's provenance from the optimizer so that the branch-free
// update stays one alignbit + one xad per word (otherwise the select that
// made `sh`/`oo` is pushed into every word).
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
    asm("" : "+v"(v));
    return v;
}

// t * K for K = 1..16 from full-rate shifts and adds.  Every intermediate
// passes through opaque(), so the optimizer cannot re-fuse the chain into a
// quarter-rate v_mul_lo_u32.
template <int K>
__device__ __forceinline__ uint32_t mul_small(uint32_t t) {
    static_assert(K >= 1 && K <= 16, "K");
    if constexpr (K == 1) return opaque(t);
    else if constexpr (K == 2 || K == 4 || K == 8 || K == 16) {
        constexpr int s = K == 2 ? 1 : K == 4 ? 2 : K == 8 ? 3 : 4;
        return opaque(t << s);
    } else if constexpr (K == 3) return opaque((t << 1) + t);
    else if constexpr (K == 5) return opaque((t << 2) + t);
    else if constexpr (K == 9) return opaque((t << 3) + t);
    else if constexpr (K == 6) return opaque(mul_small<3>(t) << 1);
    else if constexpr (K == 7) return opaque((mul_small<3>(t) << 1) + t);
    else if constexpr (K == 10) return opaque(mul_small<5>(t) << 1);
    else if constexpr (K == 11) return opaque((mul_small<5>(t) << 1) + t);
    else if constexpr (K == 12) return opaque(mul_small<3>(t) << 2);
    else if constexpr (K == 13) return opaque((mul_small<3>(t) << 2) + t);
    else if constexpr (K == 14) return opaque(mul_small<7>(t) << 1);
    else return opaque((mul_small<7>(t) << 1) + t);  // 15
}

// (t << 4) + m in one instruction.
__device__ __forceinline__ uint32_t lshl4_add(uint32_t t, uint32_t m) {
    uint32_t r;
    asm("v_lshl_add_u32 %0, %1, 4, %2" : "=v"(r) : "v"(t), "v"(m));
    return r;
}

// A uniform value (kept in an SGPR) whose provenance is hidden.  Volatile,
// so that address arithmetic derived from it is not hoisted out of the loop
// it sits in, nor shared between two places that recompute it.
__device__ __forceinline__ uint32_t opaque_s(uint32_t v) {
    asm volatile("" : "+s"(v));
    return v;
}

// `m` with a false data dependence on `after`: m cannot be formed before
// `after` is.  Used to keep one band of masks live at a time.
__device__ __forceinline__ uint32_t after_word(uint32_t m, uint32_t after) {
    asm("" : "+v"(m) : "v"(after));
    return m;
}

__device__ __forceinline__ uint32_t lane_rank(uint64_t m) {
    // number of set bits of m below this lane
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint32_t uni(uint32_t v) {
    return __builtin_amdgcn_readfirstlane(v);
}

// Global accesses as a uniform base plus a 32-bit byte offset, so that they
// compile to the scalar-base + 32-bit vector-offset form.
__device__ __forceinline__ uint32_t ld32(const uint32_t* base, uint32_t byte_off) {
    return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(base) + byte_off);
}
// NT: nontemporal (streaming) store, for data the launch never reads again.
// It raises the write bandwidth of fully written cache lines; lines that
// several wavefronts fill piecewise are better left to the normal path.
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
template <bool NT = false>
__device__ __forceinline__ void st32(uint32_t* base, uint32_t byte_off, uint32_t v) {
    uint32_t* p = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(base) + byte_off);
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}
template <bool NT = false>
__device__ __forceinline__ void st128(uint32_t* base, uint32_t byte_off, uint4 v) {
    u32x4v* p = reinterpret_cast<u32x4v*>(reinterpret_cast<char*>(base) + byte_off);
    const u32x4v x = {v.x, v.y, v.z, v.w};
    if constexpr (NT) __builtin_nontemporal_store(x, p);
    else *p = x;
}

struct RouteArgs {
    uint32_t mode;        // RC_ROUTE_MOD / RC_ROUTE_CDF
    uint32_t n_routes;    // R
    uint32_t pow2_mask;   // R - 1 when R is a power of two, else 0
    uint32_t is_pow2;
    uint32_t cdf_n;       // R - 1 thresholds
    uint32_t cdf_top;     // largest power of two <= cdf_n (0 if none)
    uint32_t guide_shift; // 32 - g (CDF mode)
    uint32_t guide_top;   // largest step of the search inside a guide bucket
};

// Route kinds, fixed per kernel instantiation.
enum : int { RK_POW2 = 0, RK_MOD = 1, RK_CDF = 2 };

// Route key: o mod R, or (CDF) from the LDS thresholds and guide table (see
// the file comment), with a branch-free search of fixed trip count.
template <int RK>
__device__ __forceinline__ uint32_t route_of(uint32_t o, const RouteArgs& ra,
                                             const uint32_t* cdf, const uint32_t* guide) {
    if constexpr (RK == RK_POW2) {
        return o & ra.pow2_mask;
    } else if constexpr (RK == RK_MOD) {
        return o % ra.n_routes;
    } else {
        const uint32_t bkt = o >> ra.guide_shift;
        uint32_t pos = guide[bkt];
        const uint32_t hi = guide[bkt + 1u];
        for (uint32_t stp = ra.guide_top; stp != 0u; stp >>= 1) {
            const uint32_t i = pos + stp;
            const uint32_t j = i < hi ? i : hi;          // min(i, hi)
            const uint32_t v = cdf[(j > 1u ? j : 1u) - 1u];  // always in range
            // both tests evaluated (no short circuit), so the read needs no
            // branch around it
            pos = ((i <= hi) & (v <= o)) ? i : pos;
        }
        return pos;
    }
}

// Route key by a plain fixed-trip binary search over all thresholds (used by
// the host-round-trip body kernel, which has no guide table).
__device__ __forceinline__ uint32_t route_of_bsearch(uint32_t o, const RouteArgs& ra,
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
    uint32_t lo = 0u;  // first lane of this lane's cohort
    if (n_coh > 1u) {
        // several sub-wavefront cohorts, listed in lane order: this lane's
        // is the last one that starts at or before it
        uint32_t at = 0u;
        for (uint32_t q = 0; q < n_coh; ++q) {
            const uint32_t cq = uni(wd[WD_LIST + q]);
            const uint32_t bq = offsets[cq];  // uniform addresses
            const uint32_t kq = offsets[cq + 1u] - bq;
            const bool mine = lane >= at;
            L.c = mine ? cq : L.c;
            b = mine ? bq : b;
            k = mine ? kq : k;
            lo = mine ? at : lo;
            at += kq;
        }
        L.s = b + (lane - lo);
    }
    L.b = b;
    L.k = k;
    L.active = lane < n_act && L.c >= cb && L.c < ce;
    L.seg = 0;
    if (!(L.flags & WF_MULTI)) {
        uint32_t hi = lo + k;
        lo = lo < 64u ? lo : 64u;
        hi = hi < 64u ? hi : 64u;
        const uint64_t below_hi = hi >= 64u ? ~0ull : ((1ull << hi) - 1ull);
        const uint64_t below_lo = lo >= 64u ? ~0ull : ((1ull << lo) - 1ull);
        L.seg = below_hi & ~below_lo;
    }
    return L;
}

// Publish this wavefront's popcount (multi-wavefront cohorts), pass the
// workgroup barrier, read the cohort's per-wavefront counts (cnt[wf .. wf+3];
// only the first nw belong to the cohort).  Called only in workgroups that
// hold a multi-wavefront cohort, the same number of times by every
// wavefront.  Publication k goes to buffer k mod 2: its readers finish
// before the barrier that follows publication k + 1, which precedes any
// write of publication k + 2.
__device__ __forceinline__ void publish_count(const LaneCohort& L, uint64_t bal, uint32_t lane,
                                              uint32_t wv, uint32_t* cnt_lds, uint32_t cnt_stride,
                                              uint32_t pub) {
    if ((L.flags & WF_MULTI) && lane == 0u)
        cnt_lds[(pub & 1u) * cnt_stride + wv] = (uint32_t)__popcll(bal);
}

// DEFER: the values are left in VGPRs and made uniform only when the slot is
// computed, so the LDS latency overlaps other work; otherwise they move to
// SGPRs at once (for kernels short of VGPRs).
template <bool DEFER = false>
__device__ __forceinline__ void barrier_read_counts(const LaneCohort& L, const uint32_t* cnt_lds,
                                                    uint32_t cnt_stride, uint32_t& pub,
                                                    uint32_t (&c4)[4]) {
    __syncthreads();
    if (L.flags & WF_MULTI) {
        const uint32_t* buf = cnt_lds + (pub & 1u) * cnt_stride + (L.flags >> 24);
#pragma unroll
        for (int i = 0; i < 4; ++i) c4[i] = DEFER ? buf[i] : uni(buf[i]);
    }
    pub += 1u;
}

__device__ __forceinline__ void exchange_counts(const LaneCohort& L, uint64_t bal, uint32_t lane,
                                                uint32_t wv, uint32_t* cnt_lds, uint32_t cnt_stride,
                                                uint32_t& pub, uint32_t (&c4)[4]) {
    publish_count(L, bal, lane, wv, cnt_lds, cnt_stride, pub);
    barrier_read_counts(L, cnt_lds, cnt_stride, pub, c4);
}

// Stable-partition slot of this lane for a step with ballot `bal`; c4 holds
// the cohort's per-wavefront counts of that step (multi-wavefront cohorts).
__device__ __forceinline__ uint32_t slot_of(const LaneCohort& L, bool dk, uint64_t bal,
                                            const uint32_t (&c4)[4], uint32_t& n1) {
    uint32_t rank_t;
    if (!(L.flags & WF_MULTI)) {
        const uint64_t bs = bal & L.seg;
        n1 = (uint32_t)__popcll(bs);
        rank_t = lane_rank(bs);
    } else {
        const uint32_t wi = (L.flags >> 8) & 0xFFu;
        const uint32_t nw = (L.flags >> 16) & 0xFFu;
        uint32_t before = 0, total = 0;
#pragma unroll
        for (uint32_t i = 0; i < 4; ++i) {
            const uint32_t ci = uni(c4[i]);
            total += (i < nw) ? ci : 0u;
            before += (i < wi) ? ci : 0u;
        }
        n1 = total;
        rank_t = before + lane_rank(bal);
    }
    const uint32_t in_c = L.s - L.b;
    return L.b + (dk ? rank_t : n1 + (in_c - rank_t));
}

// ---------------------------------------------------------------------------
// Table image (built once per handle)
// ---------------------------------------------------------------------------
struct ImageArgs {
    const uint32_t* raw;  // [R][16]
    const uint32_t* cdf;  // [R-1]
    uint32_t* img;
    uint32_t* max_span;   // out: largest guide bucket span
    uint32_t n_routes, row_words, full, tab_words, tools_off, cdf_off, cdf_n;
    uint32_t guide_off, guide_n, guide_shift, total_words;
    uint32_t m0_words, rows_off;  // full image: word-0 masks at 0, rows at rows_off
};

// number of thresholds <= x (plain binary search over global memory)
__device__ __forceinline__ uint32_t count_le(const uint32_t* cdf, uint32_t n, uint32_t x) {
    uint32_t lo = 0, hi = n;
    while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2u;
        if (cdf[mid] <= x) lo = mid + 1u; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(256) void rc_prep_kernel(ImageArgs a) {
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i >= a.total_words) return;
    const uint32_t R = a.n_routes;
    uint32_t v = 0;
    if (a.full && i < a.m0_words) {
        // word 0's taken mask of route i (row R and the padding: zero)
        if (i < R) v = a.raw[i * 16u];
    } else if (i >= a.rows_off && i < a.rows_off + a.tab_words) {
        const uint32_t j = i - a.rows_off;
        if (a.full) {
            // row r: W masks, then one zero block of padding
            const uint32_t WM = a.row_words, RS = WM + 4u;
            const uint32_t r = j / RS, w = j % RS;
            if (r < R && w < WM) v = a.raw[r * 16u + (w & 15u)] * (w + 1u);
        } else {
            const uint32_t i2 = j;
            const uint32_t r = i2 / 16u, p = i2 % 16u;
            const uint32_t q = (p >> 2) ^ (r & 3u);
            const uint32_t w = 4u * q + (p & 3u);
            if (r < R) v = a.raw[r * 16u + w];
        }
    } else if (a.full && i >= a.tools_off && i < a.tools_off + R) {
        const uint32_t r = i - a.tools_off;
        v = (a.raw[r * 16u] & 7u) | ((a.raw[r * 16u + 1u] & 7u) << 8);
    } else if (i >= a.cdf_off && i < a.cdf_off + a.cdf_n) {
        v = a.cdf[i - a.cdf_off];
    } else if (a.guide_n && i >= a.guide_off && i < a.guide_off + a.guide_n) {
        const uint32_t bkt = i - a.guide_off;
        const uint32_t last = a.guide_n - 1u;
        v = bkt == last ? a.cdf_n : count_le(a.cdf, a.cdf_n, bkt << a.guide_shift);
        if (bkt < last) {
            const uint32_t nxt = bkt + 1u == last ? a.cdf_n
                                                  : count_le(a.cdf, a.cdf_n, (bkt + 1u) << a.guide_shift);
            atomicMax(a.max_span, nxt - v);
        }
    }
    a.img[i] = v;
}

// ---------------------------------------------------------------------------
// Device-resident chain
// ---------------------------------------------------------------------------
struct ChainArgs {
    uint32_t* state;
    uint32_t* outcome;
    uint32_t* eff_sid;
    uint32_t* eff_tool;
    uint32_t* eff_payload;
    uint32_t* n_taken;
    const uint32_t* img;      // LDS image, img_words words
    const uint32_t* offsets;  // [C+1]
    const uint32_t* wdesc;    // [bins][waves][WD_WORDS]
    RouteArgs ra;
    uint32_t ld, n_words, n_cohorts, thr, step0, n_steps;
    uint32_t cohort_begin, cohort_end;
    uint32_t bins_a_lo, bins_a_n, bins_b_lo, bins_b_n;  // sub-wave / multi-wave bins
    uint32_t img_words, tools_off, cdf_off, guide_off;  // in words
    uint32_t rows_off;     // full image: first word of the mask rows
    uint32_t chain_words;  // full image: words [0, chain_words) are what the word-0 chain reads
    const uint32_t* dbits;  // no-decision floor: [T][dwords] decision bitmap
    uint32_t dwords;
};

// No-decision floor: the bitmap word holding session s's decision at chained
// step t (bit s mod 32).  Idle lanes read session 0's word.
__device__ __forceinline__ uint32_t dword_of(const ChainArgs& a, uint32_t t, uint32_t s) {
    return a.dbits[(size_t)t * a.dwords + (s >> 5)];
}

// No-decision floor, table image: session s's decisions of the 16 steps from
// t0 (bit i = step t0 + i; steps past the chain read its last step's word),
// zero for idle lanes.  One word at a time, on purpose (see the caller).
__device__ __forceinline__ uint32_t decision_block(const ChainArgs& a, const LaneCohort& L, uint32_t t0) {
    const uint32_t s = L.active ? L.s : 0u;
    uint32_t m = 0u;
#pragma unroll 1
    for (uint32_t i = 0; i < 16u; ++i) {
        const uint32_t t = t0 + i < a.n_steps ? t0 + i : a.n_steps - 1u;
        m |= ((dword_of(a, t, s) >> (s & 31u)) & 1u) << i;
    }
    return L.active ? m : 0u;
}

// One row (WM words) of the image; logical block q of row r sits at block
// q ^ (r mod NB), so its byte address is one XOR away.
template <int WM>
__device__ __forceinline__ void load_row(const uint32_t* lds, uint32_t row, uint32_t (&m)[WM]) {
    constexpr uint32_t NB = WM / 4;
    const uint32_t rb = row * (NB * 16u) + ((row & (NB - 1u)) << 4);
    const char* base = reinterpret_cast<const char*>(lds);
#pragma unroll
    for (uint32_t q = 0; q < NB; ++q) {
        const uint4 v = *reinterpret_cast<const uint4*>(base + (rb ^ (q << 4)));
        m[4 * q + 0] = v.x;
        m[4 * q + 1] = v.y;
        m[4 * q + 2] = v.z;
        m[4 * q + 3] = v.w;
    }
}

// Tool of route r for decision d: table[r][d] mod 8.
template <bool FULL>
__device__ __forceinline__ uint32_t tool_of(const uint32_t* lds, const uint32_t* lds_tools,
                                            uint32_t r, bool d) {
    if constexpr (FULL) {
        return (lds_tools[r] >> (d ? 8u : 0u)) & 7u;
    } else {
        // table[r][0..3] is block 0 of row r, stored at block (r mod 4)
        return lds[r * 16u + ((r & 3u) << 2) + (d ? 1u : 0u)] & 7u;
    }
}

// Table image, band 0 (words 4..15): masks table[r][j] * (j + 1).
template <int J, int WMAX>
__device__ __forceinline__ void band0(uint32_t (&S)[WMAX], const uint32_t (&tv)[16],
                                      uint32_t (&M)[16], uint32_t sh, uint32_t oo) {
    if constexpr (J < 16) {
        M[J] = mul_small<J + 1>(tv[J]);
        if constexpr (J < WMAX)
            S[J] = (rotr32(S[J], sh) ^ M[J]) + oo;  // words >= W: padding, see band()
        band0<J + 1, WMAX>(S, tv, M, sh, oo);
    }
}

// Table image, band B >= 1 (words 16 B .. 16 B + 15): the mask of w is the
// mask of w - 16 plus table[r][w mod 16] << 4; it is formed only after word
// w - 16 is done, so one band of masks is live at a time.
template <int B, int WMAX>
__device__ __forceinline__ void band(uint32_t (&S)[WMAX], const uint32_t (&tv)[16],
                                     uint32_t (&M)[16], uint32_t sh, uint32_t oo) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        constexpr int base = 16 * B;
        // one v_lshl_add_u32 per mask (written out, so that the shift is
        // not computed once and kept for every band)
        M[j] = after_word(lshl4_add(tv[j], M[j]), S[base + j - 16]);
        // Every word is updated, also past W: those registers start at zero,
        // are never stored, and feed nothing else, while a per-word branch
        // here would keep extra values live across the bands (and spill).
        S[base + j] = (rotr32(S[base + j], sh) ^ M[j]) + oo;
    }
}

// One bin of the resident chain.  MULTI: the bin holds cohorts of more than
// 64 sessions (every non-empty wavefront is part of one), so each step
// exchanges popcounts behind a workgroup barrier; otherwise every cohort lies
// inside one wavefront and no barrier is needed.
// FLOOR: the no-decision floor -- every decision is read from the bitmap
// (16 steps of a lane's decisions loaded at once and packed into one
// register) instead of computed; nothing else changes.
template <int WMAX, bool EXACT, int NWAVE, bool FULL, int RK, bool MULTI, bool FLOOR>
struct Chain {
    static constexpr int MW = FULL ? WMAX : 16;
    // Effect stores are nontemporal here: this path serves the large
    // variable-cohort workloads, whose bins are mostly sub-wavefront cohorts
    // that write whole lines per wavefront.
    static constexpr bool NTE = true;
    static constexpr uint32_t CNT_STRIDE = NWAVE + 4;

    // Everything one lane carries from step to step.
    struct Lane {
        uint32_t S[WMAX];
        uint32_t o, r, step, pub;
        uint32_t dm;  // FLOOR: this lane's decisions of the current 16-step block (bit i)
        bool dk;
        uint64_t bal;
        uint32_t c4[4];
    };

    // One chained step.  Full image: `mc` holds this step's masks and the
    // next step's row is prefetched into `mn`.  Table image: `mc` receives
    // this step's table row.  The next step's decision is made (and, for
    // MULTI, its popcount exchanged) even after the last step: the work is
    // discarded, and every wavefront runs the same schedule.
    static __device__ __forceinline__ void step(const ChainArgs& a, const LaneCohort& L, Lane& st,
                                                uint32_t t, uint32_t lane, uint32_t wv,
                                                const uint32_t* lds, uint32_t* lds_cnt,
                                                uint32_t (&mc)[MW], uint32_t (&mn)[MW]) {
        const uint32_t R = a.ra.n_routes;
        const uint32_t W = a.n_words;

        const uint32_t sh = opaque(st.dk ? 0u : ((31u - st.r) & 31u));
        const uint32_t oo = opaque(st.dk ? 0u : st.o);
        const uint32_t tool = tool_of<FULL>(lds, lds + a.tools_off, st.r, st.dk);
        uint32_t M[16];  // table image: running masks of the 16 columns
        if constexpr (!FULL) {
            load_row<16>(lds, st.dk ? st.r : R, mc);
            M[0] = mul_small<1>(mc[0]);
            M[1] = mul_small<2>(mc[1]);
            M[2] = mul_small<3>(mc[2]);
            M[3] = mul_small<4>(mc[3]);
        }

        // (a6) words 0..3: the payload, and the input of the next decision
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t m = FULL ? mc[w] : M[w];
            if (EXACT || (uint32_t)w < W) st.S[w] = (rotr32(st.S[w], sh) ^ m) + oo;
        }

        // (a8) chain: next outcome; (a3, a4) the next step's route and decision
        const uint32_t o_n = dev_fmix32(st.S[0]);
        const uint32_t r_n = route_of<RK>(o_n, a.ra, lds + a.cdf_off, lds + a.guide_off);
        bool d_n;
        if constexpr (FLOOR) {
            // a new 16-step block: its words, one at a time (a wait for a
            // load drains the effect stores in flight, so it happens once
            // per block, and the serial loop keeps no extra registers live)
            const uint32_t tn = t + 1u;
            if ((tn & 15u) == 0u && tn < a.n_steps) st.dm = decision_block(a, L, tn);
            d_n = L.active && ((st.dm >> (tn & 15u)) & 1u);
        } else {
            d_n = L.active && ((dev_fmix32(st.S[0] ^ o_n ^ (st.step + 1u)) & 0xFFFFu) < a.thr);
        }
        const uint64_t bal_n = __ballot(d_n);
        if constexpr (MULTI) publish_count(L, bal_n, lane, wv, lds_cnt, CNT_STRIDE, st.pub);
        if constexpr (FULL) load_row<MW>(lds, d_n ? r_n : R, mn);

        // (a6) the remaining words
        if constexpr (FULL) {
#pragma unroll
            for (int w = 4; w < WMAX; ++w)
                if (EXACT || (uint32_t)w < W) st.S[w] = (rotr32(st.S[w], sh) ^ mc[w]) + oo;
        } else {
            band0<4, WMAX>(st.S, mc, M, sh, oo);
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (WMAX > 16) {
                band<1, WMAX>(st.S, mc, M, sh, oo);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (WMAX > 32) {
                band<2, WMAX>(st.S, mc, M, sh, oo);
                __builtin_amdgcn_sched_barrier(0);
                band<3, WMAX>(st.S, mc, M, sh, oo);
            }
        }

        // the next step's counts: every wavefront has published by now
        uint32_t c4n[4] = {0u, 0u, 0u, 0u};
        if constexpr (MULTI) barrier_read_counts<FULL>(L, lds_cnt, CNT_STRIDE, st.pub, c4n);

        // (a5) compaction of this step: stable partition, taken first
        uint32_t n1, rank_t;
        if constexpr (MULTI) {
            const uint32_t wi = (L.flags >> 8) & 0xFFu;
            const uint32_t nw = (L.flags >> 16) & 0xFFu;
            uint32_t before = 0, total = 0;
#pragma unroll
            for (uint32_t i = 0; i < 4; ++i) {
                const uint32_t ci = uni(st.c4[i]);
                total += (i < nw) ? ci : 0u;
                before += (i < wi) ? ci : 0u;
            }
            n1 = total;
            rank_t = before + lane_rank(st.bal);
        } else {
            const uint64_t bs = st.bal & L.seg;
            n1 = (uint32_t)__popcll(bs);
            rank_t = lane_rank(bs);
        }
        const uint32_t in_c = L.s - L.b;
        const uint32_t slot = L.b + (st.dk ? rank_t : n1 + (in_c - rank_t));

        // (a7) emit.  slot - b < k always holds; the test keeps a compaction
        // defect from ever becoming a write outside the cohort's slots.
        if (L.active && slot - L.b < L.k) {
            const size_t slice = (size_t)t * a.ld;
            st32<NTE>(a.eff_sid + slice, slot << 2, L.s);
            st32<NTE>(a.eff_tool + slice, slot << 2, tool);
            st128<NTE>(a.eff_payload + slice * 4u, slot << 4,
                       make_uint4(st.S[0], st.S[1], st.S[2], st.S[3]));
            if (L.s == L.b) st32(a.n_taken + (size_t)t * a.n_cohorts, L.c << 2, n1);
        }

        st.o = o_n;
        st.r = r_n;
        st.dk = d_n;
        st.bal = bal_n;
#pragma unroll
        for (int i = 0; i < 4; ++i) st.c4[i] = c4n[i];
        st.step += 1u;
    }

    static __device__ __forceinline__ void run(const ChainArgs& a, uint32_t bin, uint4* lds4) {
        uint32_t* lds = reinterpret_cast<uint32_t*>(lds4);
        const uint32_t tid = threadIdx.x;
        const uint32_t lane = tid & 63u;
        const uint32_t wv = tid >> 6;
        const uint32_t W = a.n_words;
        const uint32_t R = a.ra.n_routes;
        const uint32_t T = a.n_steps;
        uint32_t* lds_cnt = lds + a.img_words;  // [2][NWAVE + 4]

        // (a1) stage the table image (eight 16-byte loads per thread in flight)
        {
            const uint4* src = reinterpret_cast<const uint4*>(a.img);
            const uint32_t n4 = a.img_words / 4u;
            constexpr uint32_t WG = NWAVE * 64;
            for (uint32_t j0 = tid; j0 < n4; j0 += 8u * WG) {
                uint4 v[8];
#pragma unroll
                for (uint32_t k = 0; k < 8; ++k) {
                    const uint32_t j = j0 + k * WG;
                    v[k] = src[j < n4 ? j : n4 - 1u];
                }
#pragma unroll
                for (uint32_t k = 0; k < 8; ++k)
                    if (j0 + k * WG < n4) lds4[j0 + k * WG] = v[k];
            }
            __syncthreads();
        }

        const LaneCohort L = lane_cohort(a.wdesc + ((size_t)bin * NWAVE + wv) * WD_WORDS,
                                         a.offsets, lane, a.cohort_begin, a.cohort_end);
        const uint32_t soff = L.s << 2;
        Lane st;
        st.pub = 0;

        // (a2) load the state words and the pending outcome
#pragma unroll
        for (int w = 0; w < WMAX; ++w) st.S[w] = 0;
        st.o = 0;
        // FLOOR: the first 16 steps' decision words, issued ahead of the
        // state words (steps past the chain read its last step's word), so
        // that the loop has no global load until step 16
        uint32_t dwd[16];
        st.dm = 0u;
        if constexpr (FLOOR) {
            const uint32_t ls = L.active ? L.s : 0u;
#pragma unroll
            for (uint32_t i = 0; i < 16u; ++i) dwd[i] = dword_of(a, i < T ? i : T - 1u, ls);
        }
        if (L.active) {
            const uint32_t ldw = opaque_s(a.ld);
            st.o = ld32(a.outcome, soff);
#pragma unroll
            for (int w = 0; w < WMAX; ++w)
                if (EXACT || (uint32_t)w < W) st.S[w] = ld32(a.state + (size_t)w * ldw, soff);
        }
        if constexpr (FLOOR) {
            uint32_t m = 0u;
#pragma unroll
            for (uint32_t i = 0; i < 16u; ++i) m |= ((dwd[i] >> (L.s & 31u)) & 1u) << i;
            st.dm = L.active ? m : 0u;
        }

        // decision of the first step
        st.step = a.step0;
        st.r = route_of<RK>(st.o, a.ra, lds + a.cdf_off, lds + a.guide_off);
        if constexpr (FLOOR)
            st.dk = (st.dm & 1u) != 0u;
        else
            st.dk = L.active && ((dev_fmix32(st.S[0] ^ st.o ^ st.step) & 0xFFFFu) < a.thr);
        st.bal = __ballot(st.dk);
#pragma unroll
        for (int k = 0; k < 4; ++k) st.c4[k] = 0u;
        if constexpr (MULTI) exchange_counts(L, st.bal, lane, wv, lds_cnt, CNT_STRIDE, st.pub, st.c4);
        uint32_t mA[MW], mB[MW];
        if constexpr (FULL) load_row<MW>(lds, st.dk ? st.r : R, mA);

        // T chained steps, unrolled by two so the prefetched row needs no copy
        for (uint32_t t = 0; t < T; t += 2u) {
            step(a, L, st, t, lane, wv, lds, lds_cnt, mA, mB);
            if (t + 1u < T) step(a, L, st, t + 1u, lane, wv, lds, lds_cnt, mB, mA);
        }

        // (a9) store the state and the next outcome (addresses recomputed
        // rather than kept live across the chain)
        if (L.active) {
            const uint32_t ldw = opaque_s(a.ld);
#pragma unroll
            for (int w = 0; w < WMAX; ++w)
                if (EXACT || (uint32_t)w < W) st32<true>(a.state + (size_t)w * ldw, soff, st.S[w]);
            st32<true>(a.outcome, soff, st.o);
        }
    }
};

// Workgroup barrier for LDS traffic only: each wavefront waits for its own
// LDS accesses (lgkmcnt 0; vmcnt and expcnt left at their maxima), not for
// its global loads and stores, which no other wavefront reads -- so state
// loads stay in flight across it.  (A workgroup release fence would wait for
// every outstanding global access as well.)
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Wait until at most N vector-memory accesses of this wavefront are
// outstanding (lgkmcnt and expcnt unconstrained).  They complete in issue
// order, so this waits for everything issued before the last N.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N <= 63, "vmcnt is a 6-bit count");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Full-image chain, split by what each word depends on.  A session's route,
// decision and next outcome at every step are functions of word 0 and the
// outcome alone; every other word only follows the per-step (mask row,
// rotation, addend) those choose.  Each chunk of up to TC steps runs as:
//   chain:   word 0 alone through the chunk -- two hashes, the route and the
//            decision per step -- recording (rotation | d << 5 | r << 6) and
//            the addend of every step; no store;
//   counts:  each wavefront publishes its taken count of every step of the
//            chunk (cohorts spanning wavefronts), then one barrier;
//   replay:  step by step, the words from the recorded control (one 16-byte
//            LDS read and two VALU ops per four words), the stable-partition
//            slot, and the effect stores.
// SPLIT: two lanes per session.  Wavefronts [0, NWAVE) ("A") run the plan's
// sessions: the chain, words [0, WA), the slots and the effects.
// Wavefronts [NWAVE, 2 NWAVE) ("B") mirror them lane for lane and replay
// words [WA, W) from the control the A lanes leave in LDS before the chunk's
// barrier; a second barrier closes the chunk when another follows.  The two
// roles run separate straight-line sequences with the same barriers.
// Rows of the mask image are W + 4 words apart (one zero block of padding
// shifts consecutive rows across the LDS banks), so block q of a row is an
// immediate offset from the row's byte offset.
// PIPED (W <= 32, WMAX = 16 or 32): three lanes per session; the A lanes
// keep only the chain and run it one 4-step chunk ahead, the B lanes replay
// words [0, 8) and emit the effects, the C lanes replay the rest (see PIPE
// below).
// FLOOR: the no-decision floor -- the A lanes read every decision from the
// bitmap instead of computing it (SPLIT: the first two chunks' words issued
// with the staging loads, later chunks' a chunk ahead).
template <int WMAX, bool EXACT, int NWAVE, int RK, bool MULTI, bool SPLIT, bool FLOOR, bool PIPED>
struct ChainF {
    static constexpr uint32_t CNT_STRIDE = NWAVE + 4;
    // Words per lane.  SPLIT: an A lane holds words [0, WA) of its session
    // and emits the effects; its B lane holds words [WA, WMAX).  At
    // WMAX = 32 the A lanes hold only the four payload words: once a
    // wavefront has issued stores, waiting for any earlier load means
    // waiting for everything on the vector-memory counter, so a lane that
    // emits effects should have no load left to wait for -- and the 28 words
    // of the B lanes then arrive while the effects go out.
    // PIPE (PIPED at WMAX = 16 or 32): three lanes per session.  The A
    // lanes hold only word 0 and the outcome and run the chain one 4-step
    // chunk ahead, storing nothing but the final outcome; behind it, the B
    // lanes replay each chunk over words [0, WP1) and emit the effects, and
    // the C lanes replay it over words [WP1, WMAX).  The chain of chunk
    // k + 1 then overlaps the replay of chunk k, where the two-role split
    // runs its 16-step chunks' chains and replays in turn; splitting the
    // replay over two roles gives it eight wavefronts per cohort to hide its
    // LDS and dependence latency.  The replay starts after one 4-step chunk,
    // so its state loads are not hidden behind a 16-step chain: with more
    // than one workgroup per CU and a one-operation route (mod R) the
    // two-role split is faster (the host decides).
    static constexpr bool PIPE = SPLIT && (WMAX == 32 || WMAX == 16) && PIPED;
    static constexpr int WP1 = 8;  // PIPE: words of the B lanes (the C lanes hold the rest)
    static constexpr int NROLE = PIPE ? 3 : SPLIT ? 2 : 1;
    static constexpr int WA = PIPE ? 0 : SPLIT ? (WMAX == 32 ? 4 : WMAX / 2) : WMAX;
    static constexpr int WB = SPLIT ? WMAX - WA : 0;
    static constexpr int WS = PIPE ? WMAX - WP1 : (WA > WB ? WA : WB);  // state registers per lane
    static constexpr int NBA = WA / 4, NBB = WB / 4;  // 16-byte blocks per lane
    static constexpr uint32_t RS = (WMAX + 4) * 4;       // row stride in bytes
    // steps per chunk (PIPE: two chunks in flight, each in its own half of
    // the 16-step control and count areas)
    static constexpr int TC = PIPE ? 4 : WMAX <= 32 ? 16 : 8;
    static constexpr uint32_t WG = NROLE * NWAVE * 64;
    static constexpr int SB = WMAX <= 32 ? (SPLIT ? 5 : 10) : (SPLIT ? 3 : 6);
    static constexpr uint32_t NLA = NWAVE * 64;  // lanes of the plan's sessions (the A lanes)
    // Bins of sub-wavefront cohorts (each cohort inside one wavefront) pass
    // their effects through an LDS stage: the lane of a session writes its
    // effect at the stage position of the lane that holds the session
    // numbered like the effect's slot, and reads back the effect whose slot
    // is its own session index -- one wavefront, so LDS order is all the
    // synchronization needed.  A wavefront's stores then cover its
    // sessions' contiguous slots, whole cache lines, and go out
    // nontemporal.  Cohorts spanning wavefronts store each effect directly
    // at its slot (an LDS exchange across wavefronts at every step costs
    // more than it saves).

    static __device__ __forceinline__ uint4 lds128(const uint32_t* lds, uint32_t byte_off) {
        return *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(lds) + byte_off);
    }

    static __device__ __forceinline__ void run(const ChainArgs& a, uint32_t bin, uint4* lds4) {
        uint32_t* lds = reinterpret_cast<uint32_t*>(lds4);
        const uint32_t tid = threadIdx.x;
        const uint32_t lane = tid & 63u;
        const uint32_t wv = uni(tid >> 6);
        // 0: A; 1: B; 2 (PIPE): C -- uniform per wavefront
        const uint32_t role = SPLIT ? uni(wv / (uint32_t)NWAVE) : 0u;
        const bool role_b = role != 0u;
        const uint32_t wa = wv - role * (uint32_t)NWAVE;      // the plan wavefront it serves
        const uint32_t alane = wa * 64u + lane;                // lane index among the A lanes
        const uint32_t wbase = PIPE ? (role == 2u ? (uint32_t)WP1 : 0u) : (role_b ? (uint32_t)WA : 0u);  // first word
        const uint32_t W = a.n_words;
        const uint32_t R = a.ra.n_routes;
        const uint32_t T = a.n_steps;
        // The host reserves 16 steps of each: counts [16][NWAVE + 4], then
        // (SPLIT) the control handed to the replaying lanes -- addends
        // [16][NLA] and control words [16][NLA] -- then the effect stage of
        // sub-wavefront bins.  PIPE uses the first 2 TC steps of the count and
        // control areas (two chunks in flight).
        static_assert(TC <= 16 && (!PIPE || 2 * TC <= 16), "LDS control and count areas hold 16 steps");
        uint32_t* lds_cnt = lds + a.img_words;
        uint32_t* lds_add = lds_cnt + 16 * CNT_STRIDE;
        uint32_t* lds_ctl = lds_add + (SPLIT ? 16 * NLA : 0);
        uint32_t* stage_w = reinterpret_cast<uint32_t*>(lds_ctl + (SPLIT ? 16 * NLA : 0));
        uint4* stage_p = reinterpret_cast<uint4*>(stage_w + NLA);
        const uint32_t* lds_tools = lds + a.tools_off;

        const uint32_t rows_b = a.rows_off * 4u;  // byte offset of the mask rows in LDS
        const LaneCohort L = lane_cohort(a.wdesc + ((size_t)bin * NWAVE + wa) * WD_WORDS,
                                         a.offsets, lane, a.cohort_begin, a.cohort_end);
        const uint32_t soff = L.s << 2;
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4* src = reinterpret_cast<const u32x4*>(a.img);
        const uint32_t n4 = a.img_words / 4u;
        // Unconditional loads (idle lanes read session 0 and never store), so
        // that no branch splits the in-order load sequence.
        uint32_t S[WS];
        const uint32_t loff = L.active ? soff : 0u;
        const uint32_t ldw = opaque_s(a.ld);
        uint32_t o = 0u;
        // Word 0 of the chain (A lanes) in a variable of its own: it is
        // loaded with the outcome before the first barrier, apart from the
        // state words that follow it.
        uint32_t s0 = 0u;
        uint32_t db[TC];   // FLOOR: the decision words of the first chunk (A lanes)
        uint32_t db1[TC];  // FLOOR, SPLIT: those of the second chunk
#pragma unroll
        for (int i = 0; i < TC; ++i) db[i] = db1[i] = 0u;
#pragma unroll
        for (int w = 0; w < WS; ++w) S[w] = 0u;
        // FLOOR: a chunk's decisions packed into one register (bit i = step
        // t0 + i), so the words die as soon as they arrive
        auto pack = [&](const uint32_t (&w)[TC]) {
            uint32_t m = 0u;
#pragma unroll
            for (int i = 0; i < TC; ++i) m |= ((w[i] >> (L.s & 31u)) & 1u) << i;
            return L.active ? m : 0u;
        };
        uint32_t dm = 0u, dm1 = 0u;
        // FLOOR: decision words, issued before the state words so that the
        // chain waits only for them and word 0
        auto load_db = [&]() {
            if constexpr (FLOOR) {
#pragma unroll
                for (int i = 0; i < TC; ++i)
                    if ((uint32_t)i < T) db[i] = dword_of(a, (uint32_t)i, L.active ? L.s : 0u);
            }
        };

        // (a1, a2) Staging.  SPLIT, A wavefronts: only what the word-0 chain
        // reads -- the chain section of the image (word-0 masks, CDF
        // thresholds, guide table), the outcome and word 0 (FLOOR: and the
        // first two chunks' decision words) -- so that the chain starts
        // after the first barrier.  SPLIT, B wavefronts (idle
        // until the chunk's control is published): the mask rows and tool
        // pairs, with direct-to-LDS loads that stay in flight across the
        // first (bare) barrier; every B lane waits for its own before the
        // barrier that precedes the first read of the rows.
        typedef __attribute__((address_space(3))) void lds_void;
        auto stage_a = [&]() {
            const uint32_t c4 = a.chain_words / 4u;
            for (uint32_t blk = wa; blk * 64u < c4; blk += NWAVE) {
                const uint32_t j = blk * 64u + lane;
                if (j < c4)
                    __builtin_amdgcn_global_load_lds((const void*)(src + j), (lds_void*)(lds4 + blk * 64u), 16, 0, 0);
            }
            o = ld32(a.outcome, loff);
            s0 = ld32(a.state, loff);
            if constexpr (FLOOR) {
                // The decision words of the first two chunks go out right
                // behind them, so that their latency overlaps the staging.
                // Steps past the chain read its last step's word: exactly
                // 2 TC loads follow, and waiting until at most that many are
                // outstanding completes everything issued before them (loads
                // retire in order).  They are packed before any store.
                asm volatile("" ::: "memory");
                const uint32_t ls = L.active ? L.s : 0u;
#pragma unroll
                for (int i = 0; i < TC; ++i) db[i] = dword_of(a, (uint32_t)i < T ? (uint32_t)i : T - 1u, ls);
#pragma unroll
                for (int i = 0; i < TC; ++i)
                    db1[i] = dword_of(a, (uint32_t)(TC + i) < T ? (uint32_t)(TC + i) : T - 1u, ls);
                asm volatile("" ::: "memory");
                wait_vmcnt<2 * TC>();  // chain section in LDS, outcome and word 0 in VGPRs
            } else {
                __builtin_amdgcn_s_waitcnt(0);  // chain section in LDS, outcome and word 0 in VGPRs
            }
        };
        auto stage_b = [&]() {
            const uint32_t c4 = a.chain_words / 4u;
            // PIPE: the B and C wavefronts share the blocks
            const uint32_t b0 = PIPE ? (role - 1u) * (uint32_t)NWAVE + wa : wa;
            constexpr uint32_t BSTR = PIPE ? 2u * NWAVE : NWAVE;
            for (uint32_t blk = b0; c4 + blk * 64u < n4; blk += BSTR) {
                const uint32_t j = c4 + blk * 64u + lane;
                if (j < n4)
                    __builtin_amdgcn_global_load_lds((const void*)(src + j), (lds_void*)(lds4 + c4 + blk * 64u),
                                                     16, 0, 0);
            }
        };
        // This lane's NW words (unconditional for idle lanes, which read
        // session 0 and never store, so that no branch splits the loads).
        auto load_words = [&](auto nw_c) {
            constexpr int NW = decltype(nw_c)::value;
#pragma unroll
            for (int w = 0; w < NW; ++w)
                if (EXACT || wbase + (uint32_t)w < W) S[w] = ld32(a.state + (size_t)(wbase + w) * ldw, loff);
        };
        // One lane per session: the first batch of the image, then the
        // outcome and the state words.  Vector-memory loads complete in
        // order, so the image batch can be written to LDS while the state
        // loads are still in flight.
        auto stage_single = [&]() {
            u32x4* dst = reinterpret_cast<u32x4*>(lds4);
            u32x4 v[SB];
#pragma unroll
            for (int k = 0; k < SB; ++k) {
                const uint32_t j = tid + (uint32_t)k * WG;
                v[k] = src[j < n4 ? j : n4 - 1u];
            }
            o = ld32(a.outcome, loff);
            load_db();
            load_words(std::integral_constant<int, WS>{});
            // Blocks past the image end repeat its last block (same value,
            // same address), so the writes need no branch either.
#pragma unroll
            for (int k = 0; k < SB; ++k) {
                const uint32_t j = tid + (uint32_t)k * WG;
                dst[j < n4 ? j : n4 - 1u] = v[k];
            }
            for (uint32_t j = tid + (uint32_t)SB * WG; j < n4; j += WG) dst[j] = src[j];
            __syncthreads();
            if constexpr (FLOOR) dm = pack(db);
            s0 = S[0];
        };

        // per-wavefront constants of the compaction
        const uint32_t in_c = L.s - L.b;
        bool f[4] = {false, false, false, false}, g[4] = {false, false, false, false};
        if constexpr (MULTI) {
            const uint32_t wi = (L.flags >> 8) & 0xFFu;
            const uint32_t nw = (L.flags >> 16) & 0xFFu;
#pragma unroll
            for (uint32_t k = 0; k < 4; ++k) {
                f[k] = k < wi;  // wavefronts of the cohort before this one
                g[k] = k < nw;  // wavefronts of the cohort
            }
        }

        uint32_t step = a.step0;
        uint32_t* p_sid = a.eff_sid;
        uint32_t* p_tool = a.eff_tool;
        uint32_t* p_pay = a.eff_payload;
        uint32_t* p_cnt = a.n_taken;

        // The chain of the chunk starting at step t0 (A lanes): records its
        // control and addends, then publishes the counts and (SPLIT) the
        // control.  Chunk 0's chain runs ahead of the chunk loop, so that no
        // wait for the state words still in flight is placed before it.
        uint32_t ctl[TC], add[TC];
        // PIPE: first step slot of the half of the control and count areas
        // that holds the chunk starting at t0 (chunks alternate halves)
        auto half_of = [&](uint32_t t0) -> uint32_t {
            return PIPE ? ((t0 / (uint32_t)TC) & 1u) * (uint32_t)TC : 0u;
        };
        auto chain_chunk = [&](uint32_t t0) {
            const uint32_t n = (T - t0) < (uint32_t)TC ? (T - t0) : (uint32_t)TC;
#pragma unroll
            for (int i = 0; i < TC; ++i) {
                ctl[i] = 0u;
                add[i] = 0u;
            }
            if (!role_b) {
                // The chain is a serial dependence through two hashes per
                // step; raised issue priority keeps it moving while other
                // wavefronts of the SIMD replay (throughput work that fills
                // the gaps).
                __builtin_amdgcn_s_setprio(3);
                if constexpr (FLOOR) {
                    if (SPLIT && t0 == (uint32_t)TC)
                        dm = dm1;  // packed before the first chunk
                    else if (t0 != 0u)
                        dm = pack(db);
                }
                // chain: word 0 only
                uint32_t r = route_of<RK>(o, a.ra, lds + a.cdf_off, lds + a.guide_off);
                uint32_t m0 = lds[r];  // taken mask of word 0 on route r (chain section)
                // Branch-free: the decision is a lane mask, and the taken and
                // not-taken forms of the update differ only in masked
                // operands (a select the compiler would otherwise turn into a
                // divergent branch on this latency-bound path).
                const uint32_t act = L.active ? 1u : 0u;
#pragma unroll
                for (int i = 0; i < TC; ++i) {
                    if ((uint32_t)i >= n) continue;
                    uint32_t dbit;
                    if constexpr (FLOOR)
                        dbit = (dm >> i) & 1u;
                    else
                        dbit = act & (uint32_t)((dev_fmix32(s0 ^ o ^ step) & 0xFFFFu) < a.thr);
                    const uint32_t dmsk = 0u - dbit;  // all ones when taken
                    const uint32_t sh = (31u - r) & 31u;
                    const uint32_t rot = sh & ~dmsk;  // rotation 0 when taken
                    const uint32_t oo = o & ~dmsk;
                    // the step's control word: the rotation (bits 0..4, also
                    // the shift operand of the rotate), the decision (bit 5),
                    // the route (bits 6..15, for the tool pair) and the LDS
                    // address of the mask row the update reads -- route r's
                    // when taken, the zero row R's when not -- in 16-byte units
                    // (bits 16..31), made here in the latency-bound chain so
                    // that every replaying lane reads its row with one shift
                    ctl[i] = rot | (dmsk & 32u) | (r << 6) |
                             (((rows_b + __umul24(dbit ? r : R, RS)) >> 4) << 16);
                    add[i] = oo;
                    s0 = (rotr32(s0, rot) ^ (m0 & dmsk)) + oo;
                    o = dev_fmix32(s0);
                    r = route_of<RK>(o, a.ra, lds + a.cdf_off, lds + a.guide_off);
                    m0 = lds[r];
                    step += 1u;
                }
                // FLOOR: the next chunk's decision words, in flight during
                // this chunk's replay (SPLIT: chunk 1's are already packed)
                if constexpr (FLOOR) {
                    if ((!SPLIT || t0 >= (uint32_t)TC) && t0 + (uint32_t)TC < T) {
#pragma unroll
                        for (int i = 0; i < TC; ++i)
                            db[i] = t0 + (uint32_t)(TC + i) < T ? dword_of(a, t0 + TC + i, L.active ? L.s : 0u) : 0u;
                    }
                }
                // counts of the chunk's steps: every lane writes the same
                // (uniform) value to the same address, so no lane mask
                const uint32_t par = half_of(t0);
                if constexpr (MULTI) {
#pragma unroll
                    for (int i = 0; i < TC; ++i)
                        lds_cnt[(par + i) * CNT_STRIDE + wa] = (uint32_t)__popcll(__ballot((ctl[i] >> 5) & 1u));
                }
                // the control for the B lanes
                if constexpr (SPLIT) {
#pragma unroll
                    for (int i = 0; i < TC; ++i) {
                        lds_ctl[(par + i) * NLA + alane] = ctl[i];
                        lds_add[(par + i) * NLA + alane] = add[i];
                    }
                }
                // The two-role split keeps the raised priority through the A
                // lanes' replay too: their effect stores then start ahead of
                // the B lanes' bulk update (measured: 100,000 sessions 18.1 ->
                // 16.9 us together with the nontemporal payloads).
                if constexpr (!SPLIT || PIPE) __builtin_amdgcn_s_setprio(0);
            }
        };

        // Replay of the chunk starting at t0 over this lane's 16-byte word
        // blocks [QLO, QHI), with (EFF: the A lanes, or the B lanes under
        // PIPE) the slots and effects, step by step.  PREF: the LDS reads of
        // step i + 1 (mask blocks and, with EFF, the tool pair) are issued
        // before step i is computed; past the chunk's last step they
        // read the zero row (valid addresses, values unused).  The step count
        // is re-read so that no per-step condition stays live across the
        // phases.
        const uint32_t my = alane;  // this lane's stage position
        auto replay = [&](uint32_t t0, auto qlo_c, auto qhi_c, auto eff_c, auto pref_c) {
            constexpr int QLO = decltype(qlo_c)::value;
            constexpr int QHI = decltype(qhi_c)::value;
            constexpr int NQ = QHI - QLO;
            constexpr bool EFF = decltype(eff_c)::value;
            constexpr bool PREF = decltype(pref_c)::value;
            const uint32_t n = (T - t0) < (uint32_t)TC ? (T - t0) : (uint32_t)TC;
            const uint32_t nr = opaque_s(n);
            const uint32_t* cq0 = lds_cnt + (L.flags >> 24) + half_of(t0) * CNT_STRIDE;
            const uint32_t qoff = (wbase + 4u * QLO) * 4u;  // byte offset of the first block in a row
            // Cohorts spanning wavefronts: the chunk's counts are all in LDS
            // before its replay starts, so each wavefront combines them once
            // per chunk, lane-parallel -- lane i holds step i's taken count
            // of the cohort (n1v) and of its wavefronts before this one
            // (prev) -- and each step takes its two values with a readlane
            // (lanes past the chunk read valid count slots, unused).
            uint32_t n1v = 0u, prev = 0u;
            if constexpr (EFF && MULTI) {
                const uint32_t* q = cq0 + (lane < (uint32_t)TC ? lane : 0u) * CNT_STRIDE;
                const uint32_t c0 = q[0], c1 = q[1], c2 = q[2], c3 = q[3];
                n1v = (g[0] ? c0 : 0u) + (g[1] ? c1 : 0u) + (g[2] ? c2 : 0u) + (g[3] ? c3 : 0u);
                prev = (f[0] ? c0 : 0u) + (f[1] ? c1 : 0u) + (f[2] ? c2 : 0u);
            }
            uint4 mc[NQ];
            uint32_t tpc = 0u;
            if constexpr (PREF) {
                const uint32_t c = ctl[0];
                const uint32_t rowoff = ((c >> 16) << 4) + qoff;
#pragma unroll
                for (int q = 0; q < NQ; ++q) mc[q] = lds128(lds, rowoff + 16u * q);
                if constexpr (EFF) tpc = lds_tools[(c >> 6) & 0x3FFu];
            }
#pragma unroll
            for (int i = 0; i < TC; ++i) {
                uint4 mn[NQ];
                uint32_t tpn = 0u;
                if constexpr (!PREF) {
                    const uint32_t c = ctl[i];
                    const uint32_t rowoff = ((c >> 16) << 4) + qoff;
#pragma unroll
                    for (int q = 0; q < NQ; ++q) mc[q] = lds128(lds, rowoff + 16u * q);
                    if constexpr (EFF) tpc = lds_tools[(c >> 6) & 0x3FFu];
                }
                if (PREF && i + 1 < TC) {
                    const uint32_t c = ctl[i + 1];
                    const uint32_t rowoff = ((c >> 16) << 4) + qoff;
#pragma unroll
                    for (int q = 0; q < NQ; ++q) mn[q] = lds128(lds, rowoff + 16u * q);
                    if constexpr (EFF) tpn = lds_tools[(c >> 6) & 0x3FFu];
                }
                if ((uint32_t)i < nr) {
                    const uint32_t c = ctl[i];
                    const uint32_t oo = add[i];
#pragma unroll
                    for (int q = 0; q < NQ; ++q) {
                        const int b = 4 * (QLO + q);
                        if (!EXACT && wbase + (uint32_t)b >= W) continue;
                        S[b] = (rotr32(S[b], c) ^ mc[q].x) + oo;
                        S[b + 1] = (rotr32(S[b + 1], c) ^ mc[q].y) + oo;
                        S[b + 2] = (rotr32(S[b + 2], c) ^ mc[q].z) + oo;
                        S[b + 3] = (rotr32(S[b + 3], c) ^ mc[q].w) + oo;
                    }
                    if constexpr (EFF) {
                        const bool dk = (c >> 5) & 1u;
                        const uint32_t tool = (tpc >> (dk ? 8u : 0u)) & 7u;

                        // (a5) stable partition, taken first
                        const uint64_t bal = __ballot(dk);
                        uint32_t n1, rank_t;
                        if constexpr (MULTI) {
                            n1 = __builtin_amdgcn_readlane(n1v, i);
                            rank_t = __builtin_amdgcn_readlane(prev, i) + lane_rank(bal);
                        } else {
                            const uint64_t bs = bal & L.seg;
                            n1 = (uint32_t)__popcll(bs);
                            rank_t = lane_rank(bs);
                        }
                        const uint32_t slot = L.b + (dk ? rank_t : n1 + (in_c - rank_t));

                        // (a7) emit; slot - b < k always holds (the test keeps
                        // a compaction defect from becoming a write outside
                        // the cohort)
                        const bool put = L.active && slot - L.b < L.k;
                        if constexpr (MULTI) {
                            // a wavefront's taken and not-taken sessions land
                            // in two contiguous slot runs, so its 16-byte
                            // payloads fill most lines whole: those go out
                            // nontemporal; the 4-byte fields, spread over more
                            // partly filled lines, through the L2
                            if (put) {
                                st32(p_sid, slot << 2, L.s);
                                st32(p_tool, slot << 2, tool);
                                st128<true>(p_pay, slot << 4, make_uint4(S[0], S[1], S[2], S[3]));
                                if (in_c == 0u) st32(p_cnt, L.c << 2, n1);
                            }
                        } else {
                            // a cohort's sessions sit in consecutive lanes,
                            // so session `slot` is held at stage position
                            // my + (slot - s); sid < 2^28 leaves room for
                            // the tool
                            if (put) {
                                const uint32_t pos = my + (slot - L.s);
                                stage_w[pos] = L.s | (tool << 28);
                                stage_p[pos] = make_uint4(S[0], S[1], S[2], S[3]);
                            }
                            asm volatile("" ::: "memory");
                            if (L.active) {
                                const uint32_t w = stage_w[my];
                                const uint4 pv = stage_p[my];
                                st32<true>(p_sid, soff, w & 0x0FFFFFFFu);
                                st32<true>(p_tool, soff, w >> 28);
                                st128<true>(p_pay, soff << 2, pv);
                                if (in_c == 0u) st32(p_cnt, L.c << 2, n1);
                            }
                            asm volatile("" ::: "memory");  // this step's reads before the next step's writes
                        }
                        p_sid += ldw;
                        p_tool += ldw;
                        p_pay += 4u * ldw;
                        p_cnt += a.n_cohorts;
                    }
                }
                if (PREF && i + 1 < TC) {
#pragma unroll
                    for (int q = 0; q < NQ; ++q) mc[q] = mn[q];
                    if constexpr (EFF) tpc = tpn;
                }
            }
        };

        // (a9) store this lane's NW words and (A lanes) the next outcome (the
        // row addresses are recomputed from a fresh copy of ld rather than
        // kept live across the chain)
        auto store_state = [&](auto nw_c, bool with_outcome) {
            constexpr int NW = decltype(nw_c)::value;
            if (L.active) {
                const uint32_t ld_st = opaque_s(a.ld);
#pragma unroll
                for (int w = 0; w < NW; ++w)
                    if (EXACT || wbase + (uint32_t)w < W) st32<true>(a.state + (size_t)(wbase + w) * ld_st, soff, S[w]);
                if (with_outcome) st32<true>(a.outcome, soff, o);
            }
        };
        auto bare_barrier = []() {
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        };
        using Z = std::integral_constant<int, 0>;
        using NA = std::integral_constant<int, NBA>;
        using NB = std::integral_constant<int, NBB>;
        using Yes = std::integral_constant<bool, true>;
        using No = std::integral_constant<bool, false>;
        // the B lanes of a 28-word split read each step's masks when the step
        // starts (no room for a second set of mask registers)
        using PrefB = std::integral_constant<bool, (NBB <= 4)>;

        // Each role runs its own straight-line sequence to the end, with the
        // same barriers per chunk, so that the compiler's wait analysis sees
        // one role's accesses at a time.  Chunk 0 runs outside the chunk
        // loop: the compiler flushes every outstanding vector-memory access
        // in the preheader of a loop that stores without loading.
        if constexpr (PIPE) {
            // The same barriers in both roles: a bare one after staging, then
            // one per chunk.  Barrier k + 1 publishes chunk k's control and
            // counts (A) and closes the replay of chunk k - 1 (B); chunk k + 2
            // reuses chunk k's half only after barrier k + 2, when its replay
            // is done.
            if (!role_b) {
                stage_a();
                bare_barrier();
                if constexpr (FLOOR) {
                    dm = pack(db);
                    dm1 = pack(db1);
                }
                for (uint32_t t0 = 0; t0 < T; t0 += TC) {
                    chain_chunk(t0);
                    lds_barrier();
                }
                if (L.active) st32<true>(a.outcome, soff, o);
            } else {
                stage_b();
                bare_barrier();
                auto read_ctl = [&](uint32_t t0) {
                    const uint32_t par = half_of(t0);
#pragma unroll
                    for (int i = 0; i < TC; ++i) {
                        ctl[i] = lds_ctl[(par + i) * NLA + alane];
                        add[i] = lds_add[(par + i) * NLA + alane];
                    }
                };
                // B (words [0, WP1), effects) and C (the rest): the same
                // barriers, each with its own straight-line sequence
                auto replay_role = [&](auto nw_c, auto nq_c, auto eff_c) {
                    constexpr int NWR = decltype(nw_c)::value;
                    load_words(nw_c);
                    // the row loads issued before the NWR state loads have
                    // landed (with W < WMAX fewer were issued: wait for all)
                    wait_vmcnt<EXACT ? NWR : 0>();
                    lds_barrier();
                    read_ctl(0u);
                    wait_vmcnt<0>();  // every word is needed at the first step
                    replay(0u, Z{}, nq_c, eff_c, No{});
                    for (uint32_t t0 = TC; t0 < T; t0 += TC) {
                        lds_barrier();
                        read_ctl(t0);
                        replay(t0, Z{}, nq_c, eff_c, No{});
                    }
                    store_state(nw_c, false);
                };
                if (role == 1u)
                    replay_role(std::integral_constant<int, WP1>{}, std::integral_constant<int, WP1 / 4>{}, Yes{});
                else
                    replay_role(std::integral_constant<int, WMAX - WP1>{},
                                std::integral_constant<int, (WMAX - WP1) / 4>{}, No{});
            }
        } else if constexpr (SPLIT) {
            if (!role_b) {
                stage_a();
                bare_barrier();
                // FLOOR: the decision words of the first two chunks (issued in
                // stage_a) are packed before any store is issued: once stores
                // are outstanding, waiting for a load drains them too.
                load_words(std::integral_constant<int, WA>{});
                if constexpr (FLOOR) {
                    dm = pack(db);
                    dm1 = pack(db1);
                }
                chain_chunk(0u);
                lds_barrier();  // publishes chunk 0's counts and control
                // The replay needs all WA words at its first step; an explicit
                // wait here (nothing else is outstanding) keeps the compiler
                // from repeating it, step after step, behind the effect stores.
                wait_vmcnt<0>();
                replay(0u, Z{}, NA{}, Yes{}, Yes{});
                for (uint32_t t0 = TC; t0 < T; t0 += TC) {
                    lds_barrier();  // every wavefront is done with the previous chunk's
                    chain_chunk(t0);
                    lds_barrier();
                    replay(t0, Z{}, NA{}, Yes{}, Yes{});
                }
                store_state(std::integral_constant<int, WA>{}, true);
            } else {
                stage_b();
                bare_barrier();
                load_words(std::integral_constant<int, WB>{});
                // the row loads issued before the WB state loads have landed
                // (with W < WMAX fewer state loads were issued: wait for all)
                wait_vmcnt<EXACT ? WB : 0>();
                lds_barrier();
                auto read_ctl = [&]() {
#pragma unroll
                    for (int i = 0; i < TC; ++i) {
                        ctl[i] = lds_ctl[i * NLA + alane];
                        add[i] = lds_add[i * NLA + alane];
                    }
                };
                read_ctl();
                wait_vmcnt<0>();  // every word is needed at the first step
                replay(0u, Z{}, NB{}, No{}, PrefB{});
                for (uint32_t t0 = TC; t0 < T; t0 += TC) {
                    lds_barrier();
                    lds_barrier();
                    read_ctl();
                    replay(t0, Z{}, NB{}, No{}, PrefB{});
                }
                store_state(std::integral_constant<int, WB>{}, false);
            }
        } else {
            stage_single();
            chain_chunk(0u);
            if constexpr (MULTI) lds_barrier();
            replay(0u, Z{}, NA{}, Yes{}, Yes{});
            for (uint32_t t0 = TC; t0 < T; t0 += TC) {
                if constexpr (MULTI) lds_barrier();
                chain_chunk(t0);
                if constexpr (MULTI) lds_barrier();
                replay(t0, Z{}, NA{}, Yes{}, Yes{});
            }
            store_state(std::integral_constant<int, WMAX>{}, true);
        }
    }
};

// One workgroup per bin: blocks [0, bins_a_n) take the sub-wavefront bins,
// the rest the multi-wavefront bins.  The table-image chain and the two-role
// full-image chain at W = 32 run two 512-lane workgroups per CU, so they are
// held to four wavefronts per SIMD (at most 128 VGPRs); the pipelined split
// (W = 16 or 32) runs two 768-lane workgroups per CU, six wavefronts per
// SIMD (at most 80 VGPRs).  At W = 64 the two-role full-image chain needs
// more registers and runs one workgroup per CU.
template <int WMAX, bool EXACT, int NWAVE, bool FULL, int RK, bool FLOOR, bool PIPED>
__global__ __launch_bounds__((FULL && (WMAX >= 32 || (PIPED && WMAX == 16)) ? (PIPED && WMAX <= 32 ? 3 : 2) : 1) *
                                 NWAVE * 64,
                             (!FULL || WMAX == 32) ? (PIPED && FULL && WMAX == 32 ? 6 : 4)
                                                   : (PIPED && WMAX == 16 ? 6 : 1))
void rc_chain_kernel(ChainArgs a) {
    extern __shared__ uint4 lds4[];
    if constexpr (FULL) {
        constexpr bool SPLIT = WMAX >= 32 || (PIPED && WMAX == 16);
        if (blockIdx.x < a.bins_a_n)
            ChainF<WMAX, EXACT, NWAVE, RK, false, SPLIT, FLOOR, PIPED>::run(a, a.bins_a_lo + blockIdx.x, lds4);
        else
            ChainF<WMAX, EXACT, NWAVE, RK, true, SPLIT, FLOOR, PIPED>::run(a, a.bins_b_lo + (blockIdx.x - a.bins_a_n), lds4);
    } else {
        if (blockIdx.x < a.bins_a_n)
            Chain<WMAX, EXACT, NWAVE, FULL, RK, false, FLOOR>::run(a, a.bins_a_lo + blockIdx.x, lds4);
        else
            Chain<WMAX, EXACT, NWAVE, FULL, RK, true, FLOOR>::run(a, a.bins_b_lo + (blockIdx.x - a.bins_a_n), lds4);
    }
}

// ---------------------------------------------------------------------------
// Host round trip
// ---------------------------------------------------------------------------

// Part 1: decide and compact one step.  Writes n_taken and, for every
// stepped session, perm[slot] = sid | d << 31 (the stable partition of each
// cohort, in effect order), and adds the workgroup's taken count to
// ctr[parity] (the 4-byte word the host reads), one global atomic per
// workgroup.  Block 0 clears the other parity's counter for the next step.
struct DecideArgs {
    const uint32_t* state;
    const uint32_t* outcome;
    uint32_t* n_taken;
    uint32_t* perm;           // slot j of the stepped range at perm[j - perm_lo]
    uint32_t* ctr;            // [2]
    const uint32_t* offsets;
    const uint32_t* wdesc;
    uint32_t thr, step, t_index, n_cohorts, n_sessions;
    uint32_t cohort_begin, cohort_end;
    uint32_t bins_a_lo, bins_a_n, bins_b_lo, parity, perm_lo;
};

template <int NWAVE>
__global__ __launch_bounds__(NWAVE * 64) void rc_decide_kernel(DecideArgs a) {
    __shared__ uint32_t cnt_lds[2 * (NWAVE + 4)];
    __shared__ uint32_t wg_taken;
    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63u;
    const uint32_t wv = tid >> 6;
    if (tid == 0u) {
        wg_taken = 0u;
        if (blockIdx.x == 0u) a.ctr[a.parity ^ 1u] = 0u;
    }
    const uint32_t i = blockIdx.x;
    const uint32_t bin = i < a.bins_a_n ? a.bins_a_lo + i : a.bins_b_lo + (i - a.bins_a_n);
    const LaneCohort L = lane_cohort(a.wdesc + ((size_t)bin * NWAVE + wv) * WD_WORDS,
                                     a.offsets, lane, a.cohort_begin, a.cohort_end);
    uint32_t s0w = 0, o = 0;
    if (L.active) {
        s0w = ld32(a.state, L.s << 2);
        o = ld32(a.outcome, L.s << 2);
    }
    const bool dk = L.active && ((dev_fmix32(s0w ^ o ^ a.step) & 0xFFFFu) < a.thr);
    const uint64_t bal = __ballot(dk);
    uint32_t c4[4] = {0u, 0u, 0u, 0u};
    uint32_t pub = 0;
    __syncthreads();  // wg_taken is cleared
    if (L.flags & WF_WGMULTI) exchange_counts(L, bal, lane, wv, cnt_lds, NWAVE + 4, pub, c4);
    uint32_t n1;
    const uint32_t slot = slot_of(L, dk, bal, c4, n1);
    if (L.active && L.s == L.b) a.n_taken[(size_t)a.t_index * a.n_cohorts + L.c] = n1;
    if (L.active && slot - L.b < L.k) a.perm[slot - a.perm_lo] = L.s | (dk ? 0x80000000u : 0u);
    if (lane == 0u && bal) atomicAdd(&wg_taken, (uint32_t)__popcll(bal));
    __syncthreads();
    if (tid == 0u && wg_taken) atomicAdd(&a.ctr[a.parity], wg_taken);
}

// Part 2: the route body the host selected.  Walks the slots [lo, hi) of
// the stepped cohorts and handles the sessions of its own population, with
// the slot the decide kernel assigned.
struct BodyArgs {
    uint32_t* state;
    uint32_t* outcome;
    uint32_t* eff_sid;
    uint32_t* eff_tool;
    uint32_t* eff_payload;
    const uint32_t* perm;  // slot j at perm[j - lo]
    const uint32_t* raw;   // [R][16]
    const uint32_t* cdf;
    RouteArgs ra;
    uint32_t ld, n_words, lo, hi, t_index, n_sessions;
};

template <int WMAX, bool EXACT, bool TAKEN>
__global__ __launch_bounds__(256) void rc_body_kernel(BodyArgs a) {
    __shared__ uint32_t cdf_lds[RC_MAX_ROUTES];
    const uint32_t tid = threadIdx.x;
    if (a.ra.mode == RC_ROUTE_CDF) {
        for (uint32_t i = tid; i < a.ra.cdf_n; i += 256u) cdf_lds[i] = a.cdf[i];
        __syncthreads();
    }
    const uint32_t slot = a.lo + blockIdx.x * 256u + tid;
    if (slot >= a.hi) return;
    const uint32_t e = a.perm[slot - a.lo];
    if ((e >> 31) != (TAKEN ? 1u : 0u)) return;
    const uint32_t s = e & 0x7FFFFFFFu;
    if (s >= a.n_sessions) return;  // never taken by a valid permutation
    const uint32_t W = a.n_words;
    const uint32_t soff = s << 2;
    const uint32_t o = ld32(a.outcome, soff);
    const uint32_t r = route_of_bsearch(o, a.ra, cdf_lds);
    uint32_t S[WMAX];
#pragma unroll
    for (int w = 0; w < WMAX; ++w)
        S[w] = (EXACT || (uint32_t)w < W) ? ld32(a.state + (size_t)w * a.ld, soff) : 0u;
    if (TAKEN) {
        const uint32_t* row = a.raw + r * 16u;
#pragma unroll
        for (int w = 0; w < WMAX; ++w) S[w] ^= row[w & 15] * (uint32_t)(w + 1);
    } else {
        const uint32_t sh = (31u - r) & 31u;
#pragma unroll
        for (int w = 0; w < WMAX; ++w) S[w] = rotr32(S[w], sh) + o;
    }
#pragma unroll
    for (int w = 0; w < WMAX; ++w)
        if (EXACT || (uint32_t)w < W) st32(a.state + (size_t)w * a.ld, soff, S[w]);
    const size_t slice = (size_t)a.t_index * a.ld;
    st32(a.eff_sid + slice, slot << 2, s);
    st32(a.eff_tool + slice, slot << 2, (a.raw[r * 16u + (TAKEN ? 1u : 0u)]) & 7u);
    st128(a.eff_payload + slice * 4u, slot << 4, make_uint4(S[0], S[1], S[2], S[3]));
    st32(a.outcome, soff, dev_fmix32(S[0]));
}

// Clears n words (a kernel rather than a memset, so that callers that
// capture the work into a graph record no memset node).
__global__ __launch_bounds__(64) void rc_clear_kernel(uint32_t* p, uint32_t n) {
    const uint32_t i = blockIdx.x * 64u + threadIdx.x;
    if (i < n) p[i] = 0u;
}

// Scratch of rc_cohort_run_chain_noalloc: two counter words, padding, then
// the slot-to-session permutation of at most RC_NOALLOC_MAX_SESSIONS
// sessions.  Each device holds its own copy for the life of the process.
constexpr uint32_t NOALLOC_PERM_OFF = 64u;
__device__ __align__(256) uint32_t rc_noalloc_scratch[NOALLOC_PERM_OFF + RC_NOALLOC_MAX_SESSIONS];

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

typedef void (*ChainFn)(ChainArgs);
typedef void (*DecideFn)(DecideArgs);
typedef void (*BodyFn)(BodyArgs);

// The pipelined split exists for the full image at WMAX = 16 and 32.
bool has_piped(uint32_t wmax, bool full) { return full && (wmax == 32u || wmax == 16u); }

template <int WMAX, bool EXACT, int RK, bool FLOOR>
ChainFn chain_fn(bool full, bool piped) {
    if (!full) {
        if constexpr (WMAX >= 32) return rc_chain_kernel<WMAX, EXACT, 8, false, RK, FLOOR, false>;
        return nullptr;
    }
    if constexpr (WMAX == 32 || WMAX == 16)
        if (piped) return rc_chain_kernel<WMAX, EXACT, 4, true, RK, FLOOR, true>;
    return rc_chain_kernel<WMAX, EXACT, 4, true, RK, FLOOR, false>;
}

template <int WMAX, bool EXACT, bool FLOOR>
ChainFn chain_fn_rk(bool full, bool piped, int rk) {
    return rk == RK_POW2 ? chain_fn<WMAX, EXACT, RK_POW2, FLOOR>(full, piped)
         : rk == RK_MOD ? chain_fn<WMAX, EXACT, RK_MOD, FLOOR>(full, piped)
                        : chain_fn<WMAX, EXACT, RK_CDF, FLOOR>(full, piped);
}

template <bool FLOOR>
ChainFn pick_chain_t(uint32_t wmax, bool exact, bool full, bool piped, int rk) {
    switch (wmax) {
        case 4: return exact ? chain_fn_rk<4, true, FLOOR>(full, piped, rk) : chain_fn_rk<4, false, FLOOR>(full, piped, rk);
        case 8: return exact ? chain_fn_rk<8, true, FLOOR>(full, piped, rk) : chain_fn_rk<8, false, FLOOR>(full, piped, rk);
        case 16: return exact ? chain_fn_rk<16, true, FLOOR>(full, piped, rk) : chain_fn_rk<16, false, FLOOR>(full, piped, rk);
        case 32: return exact ? chain_fn_rk<32, true, FLOOR>(full, piped, rk) : chain_fn_rk<32, false, FLOOR>(full, piped, rk);
        default: return exact ? chain_fn_rk<64, true, FLOOR>(full, piped, rk) : chain_fn_rk<64, false, FLOOR>(full, piped, rk);
    }
}

ChainFn pick_chain(uint32_t wmax, bool exact, bool full, bool piped, int rk, bool floor) {
    return floor ? pick_chain_t<true>(wmax, exact, full, piped, rk)
                 : pick_chain_t<false>(wmax, exact, full, piped, rk);
}

// The pipelined split for a launch: at most one workgroup per CU, or a
// chain whose route is a threshold search (CDF mode), whose longer step
// makes the overlap pay at any launch size.  Measured on MI355X
// (256-session cohorts, W = 32, every launch streaming from HBM): 4-15%
// faster than the two-role split from 1 to 256 workgroups with mod-R
// routes, 5-27% faster at every size with CDF routes; with mod-R routes
// beyond one workgroup per CU it ties or loses (the 100,000-session chain:
// 16.3-16.6 against 14.8-15.4 us).  At W = 16 against the one-lane chain
// (64-session cohorts, T = 8, mod-16 routes): one cohort 6.42 -> 4.82 us,
// 1,000 cohorts in 250 workgroups 8.55 -> 6.5 us.
bool use_piped(uint32_t wmax, bool full, int route_kind, uint32_t grid, uint32_t n_cu) {
    return has_piped(wmax, full) && (grid <= n_cu || route_kind == RK_CDF);
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

uint32_t ceil_log2(uint32_t x) {
    uint32_t g = 0;
    while ((1u << g) < x) ++g;
    return g;
}

// Validated buffer sets remembered per handle (see validate_buffers).
constexpr int EXTENT_CACHE = 16;
struct BufferKey {
    const void* p[7];
    uint64_t bytes[7];
    bool operator==(const BufferKey& o) const {
        for (int i = 0; i < 7; ++i)
            if (p[i] != o.p[i] || bytes[i] != o.bytes[i]) return false;
        return true;
    }
};

}  // namespace

struct rc_cohort {
    int device = -1;
    uint32_t N = 0, W = 0, R = 0, C = 0, thr = 0;
    RouteArgs ra{};
    uint32_t wmax = 4;
    bool exact = true;
    bool full = true;
    int route_kind = 0;  // RK_POW2 / RK_MOD / RK_CDF
    uint32_t nwave = 4;
    uint32_t img_words = 0, tools_off = 0, cdf_off = 0, guide_off = 0, rows_off = 0, chain_words = 0;
    size_t chain_lds_bytes = 0;
    uint32_t chain_threads = 256;  // threads of a chain workgroup
    std::vector<uint32_t> offsets;  // host copy [C+1]
    Plan plan;
    uint32_t* d_offsets = nullptr;
    uint32_t* d_raw = nullptr;
    uint32_t* d_cdf = nullptr;
    uint32_t* d_img = nullptr;
    uint32_t* d_span = nullptr;
    uint32_t* d_wdesc = nullptr;
    uint32_t* d_perm = nullptr;  // host round trip: [N] slot -> sid | d << 31
    uint32_t* d_ctr = nullptr;
    uint32_t* h_word = nullptr;  // pinned
    uint32_t parity = 0;
    bool ctr_dirty = false;
    uint32_t last_launches = 0, last_d2h = 0;
    // Recorded after the last body kernel of a host-round-trip call; the next
    // such call's stream waits for it before touching d_perm / d_ctr.
    hipEvent_t hrt_done = nullptr;
    bool hrt_pending = false;
    uint32_t n_cu = 256;             // compute units of the device
    size_t lds_per_cu = 160u * 1024u;
    BufferKey seen[EXTENT_CACHE];    // buffer sets that passed the device checks
    int n_seen = 0, next_seen = 0;
};

namespace {

void free_handle(rc_cohort* h) {
    if (!h) return;
    if (h->device >= 0) {
        DeviceGuard g(h->device);
        (void)hipFree(h->d_offsets);
        (void)hipFree(h->d_raw);
        (void)hipFree(h->d_cdf);
        (void)hipFree(h->d_img);
        (void)hipFree(h->d_span);
        (void)hipFree(h->d_wdesc);
        (void)hipFree(h->d_perm);
        (void)hipFree(h->d_ctr);
        if (h->h_word) (void)hipHostFree(h->h_word);
        if (h->hrt_done) (void)hipEventDestroy(h->hrt_done);
    }
    delete h;
}

// Per device: the address of rc_noalloc_scratch (resolved once, with the
// device current) and the event that orders the no-allocation
// host-round-trip calls that share it.
constexpr int MAX_DEVICES = 64;
std::mutex g_noalloc_mu;
uint32_t* g_noalloc_ptr[MAX_DEVICES] = {};
hipEvent_t g_noalloc_done[MAX_DEVICES] = {};
bool g_noalloc_pending[MAX_DEVICES] = {};

// Called by rc_cohort_create with `dev` current.
int noalloc_init(int dev) {
    if (dev < 0 || dev >= MAX_DEVICES) return RC_E_DEVICE;
    std::lock_guard<std::mutex> lk(g_noalloc_mu);
    if (g_noalloc_ptr[dev]) return RC_OK;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(rc_noalloc_scratch)) != hipSuccess || !ptr) {
        (void)hipGetLastError();
        return RC_E_DEVICE;
    }
    hipEvent_t ev = nullptr;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();
        return RC_E_DEVICE;
    }
    g_noalloc_done[dev] = ev;
    g_noalloc_ptr[dev] = static_cast<uint32_t*>(ptr);
    return RC_OK;
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

// The caller's buffers (and, for the no-decision floor, its decision
// bitmap): present, pairwise disjoint, and each inside one device allocation
// of the handle's device.  The allocation check queries the HIP runtime; a
// buffer set (pointers and extents) that passed it is remembered, and the
// last EXTENT_CACHE such sets are not queried again.
int validate_buffers(rc_cohort* h, const rc_buffers* b, uint32_t T, bool floor = false,
                     const uint32_t* dbits = nullptr) {
    if (!b) return RC_E_INVALID;
    if (b->ld < h->N || b->ld > RC_MAX_SESSIONS) return RC_E_INVALID;
    const uint64_t ld = b->ld;
    struct Ext { const void* p; uint64_t bytes; } ext[7] = {
        {b->state, 4ull * h->W * ld},
        {b->outcome, 4ull * ld},
        {b->eff_sid, 4ull * T * ld},
        {b->eff_tool, 4ull * T * ld},
        {b->eff_payload, 16ull * T * ld},
        {b->n_taken, 4ull * T * h->C},
        {dbits, 4ull * T * ((ld + 31u) / 32u)},
    };
    const int n = floor ? 7 : 6;
    for (int i = 0; i < n; ++i) {
        if (!ext[i].p) return RC_E_INVALID;
        if (ext[i].bytes >= (1ull << 46)) return RC_E_INVALID;
    }
    for (int i = 0; i < n; ++i)
        for (int j = i + 1; j < n; ++j) {
            const uintptr_t a0 = (uintptr_t)ext[i].p, a1 = a0 + ext[i].bytes;
            const uintptr_t b0 = (uintptr_t)ext[j].p, b1 = b0 + ext[j].bytes;
            if (a0 < b1 && b0 < a1) return RC_E_INVALID;
        }
    BufferKey key;
    for (int i = 0; i < 7; ++i) {
        key.p[i] = i < n ? ext[i].p : nullptr;
        key.bytes[i] = i < n ? ext[i].bytes : 0u;
    }
    for (int i = 0; i < h->n_seen; ++i)
        if (h->seen[i] == key) return RC_OK;
    for (int i = 0; i < n; ++i)
        if (ext[i].bytes && !device_extent_ok(ext[i].p, ext[i].bytes, h->device)) return RC_E_INVALID;
    h->seen[h->next_seen] = key;
    h->next_seen = (h->next_seen + 1) % EXTENT_CACHE;
    if (h->n_seen < EXTENT_CACHE) ++h->n_seen;
    return RC_OK;
}

int launch_ok() {
    return hipGetLastError() == hipSuccess ? RC_OK : RC_E_DEVICE;
}

int run_resident(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t T,
                 uint32_t cb, uint32_t ce, hipStream_t stream, const uint32_t* dbits = nullptr) {
    ChainArgs a;
    a.state = b->state;
    a.outcome = b->outcome;
    a.eff_sid = b->eff_sid;
    a.eff_tool = b->eff_tool;
    a.eff_payload = b->eff_payload;
    a.n_taken = b->n_taken;
    a.img = h->d_img;
    a.offsets = h->d_offsets;
    a.wdesc = h->d_wdesc;
    a.ra = h->ra;
    a.ld = b->ld;
    a.n_words = h->W;
    a.n_cohorts = h->C;
    a.thr = h->thr;
    a.step0 = step0;
    a.n_steps = T;
    a.cohort_begin = cb;
    a.cohort_end = ce;
    bins_of_range(h->plan, cb, ce, a.bins_a_lo, a.bins_a_n, a.bins_b_lo, a.bins_b_n);
    a.img_words = h->img_words;
    a.tools_off = h->tools_off;
    a.cdf_off = h->cdf_off;
    a.guide_off = h->guide_off;
    a.rows_off = h->rows_off;
    a.chain_words = h->chain_words;
    a.dbits = dbits;
    a.dwords = (b->ld + 31u) / 32u;
    const uint32_t grid = a.bins_a_n + a.bins_b_n;  // one workgroup per bin
    const bool piped = use_piped(h->wmax, h->full, h->route_kind, grid, h->n_cu);
    ChainFn fn = pick_chain(h->wmax, h->exact, h->full, piped, h->route_kind, dbits != nullptr);
    // the pipelined split runs three lanes per session, the two-role split two
    hipLaunchKernelGGL(fn, dim3(grid), dim3(piped ? 3u * 64u * h->nwave : h->chain_threads), h->chain_lds_bytes,
                       stream, a);
    if (launch_ok() != RC_OK) return RC_E_DEVICE;
    h->last_launches = 1;
    h->last_d2h = 0;
    return RC_OK;
}

// Where a host-round-trip call keeps its per-step scratch: the
// slot-to-session permutation of the stepped range (slot j at
// perm[j - lo]) and the two counter words of the 4-byte observation, plus
// the event that orders the calls sharing them.
struct HrtScratch {
    uint32_t* perm;
    uint32_t* ctr;
    uint32_t* parity;   // which counter word the next step adds to
    hipEvent_t done;    // recorded after a call's last body kernel
    bool* pending;      // `done` has been recorded
    bool clear_first;   // clear both counter words with a kernel first
};

int run_host_roundtrip(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t T,
                       uint32_t cb, uint32_t ce, hipStream_t stream, const HrtScratch& sc) {
    uint32_t launches = 0, copies = 0;
    // the previous call that used this scratch may still be running on
    // another stream: wait for its last body kernel
    if (*sc.pending && hipStreamWaitEvent(stream, sc.done, 0) != hipSuccess) return RC_E_DEVICE;
    if (sc.clear_first) {
        hipLaunchKernelGGL(rc_clear_kernel, dim3(1), dim3(64), 0, stream, sc.ctr, 2u);
        if (launch_ok() != RC_OK) return RC_E_DEVICE;
        ++launches;
        *sc.parity = 0;
    }
    uint32_t a_lo, a_n, b_lo, b_n;
    bins_of_range(h->plan, cb, ce, a_lo, a_n, b_lo, b_n);
    const uint32_t grid = a_n + b_n;
    const uint32_t lo = h->offsets[cb], hi = h->offsets[ce];
    const uint32_t n_range = hi - lo;
    const uint32_t body_grid = (n_range + 255u) / 256u;
    DecideFn dfn = pick_decide(h->nwave);
    BodyFn taken_fn = pick_body(h->wmax, h->exact, true);
    BodyFn not_fn = pick_body(h->wmax, h->exact, false);
    for (uint32_t t = 0; t < T; ++t) {
        if (!sc.clear_first) h->ctr_dirty = true;  // the handle's counters; cleared again when the step completes
        DecideArgs d;
        d.state = b->state;
        d.outcome = b->outcome;
        d.n_taken = b->n_taken;
        d.perm = sc.perm;
        d.ctr = sc.ctr;
        d.offsets = h->d_offsets;
        d.wdesc = h->d_wdesc;
        d.thr = h->thr;
        d.step = step0 + t;
        d.t_index = t;
        d.n_cohorts = h->C;
        d.n_sessions = h->N;
        d.cohort_begin = cb;
        d.cohort_end = ce;
        d.bins_a_lo = a_lo;
        d.bins_a_n = a_n;
        d.bins_b_lo = b_lo;
        d.parity = *sc.parity;
        d.perm_lo = lo;
        hipLaunchKernelGGL(dfn, dim3(grid), dim3(h->nwave * 64), 0, stream, d);
        if (launch_ok() != RC_OK) return RC_E_DEVICE;
        ++launches;
        // the observation: 4 bytes to pinned host memory, then wait
        if (hipMemcpyAsync(h->h_word, sc.ctr + *sc.parity, sizeof(uint32_t),
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
        ba.perm = sc.perm;
        ba.raw = h->d_raw;
        ba.cdf = h->d_cdf;
        ba.ra = h->ra;
        ba.ld = b->ld;
        ba.n_words = h->W;
        ba.lo = lo;
        ba.hi = hi;
        ba.t_index = t;
        ba.n_sessions = h->N;
        if (n_taken_total > 0u) {
            hipLaunchKernelGGL(taken_fn, dim3(body_grid), dim3(256), 0, stream, ba);
            if (launch_ok() != RC_OK) return RC_E_DEVICE;
            ++launches;
        }
        if (n_taken_total < n_range) {
            hipLaunchKernelGGL(not_fn, dim3(body_grid), dim3(256), 0, stream, ba);
            if (launch_ok() != RC_OK) return RC_E_DEVICE;
            ++launches;
        }
        *sc.parity ^= 1u;
        if (!sc.clear_first) h->ctr_dirty = false;
    }
    if (hipEventRecord(sc.done, stream) != hipSuccess) return RC_E_DEVICE;
    *sc.pending = true;
    h->last_launches = launches;
    h->last_d2h = copies;
    return RC_OK;
}

// The handle's own scratch (d_perm, d_ctr), after restoring cleared counters
// if a previous call stopped inside a step.
int run_host_roundtrip_handle(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t T,
                              uint32_t cb, uint32_t ce, hipStream_t stream) {
    if (h->ctr_dirty) {
        if (h->hrt_pending && hipStreamWaitEvent(stream, h->hrt_done, 0) != hipSuccess) return RC_E_DEVICE;
        if (hipMemsetAsync(h->d_ctr, 0, 2 * sizeof(uint32_t), stream) != hipSuccess) return RC_E_DEVICE;
        h->parity = 0;
        h->ctr_dirty = false;
    }
    HrtScratch sc{h->d_perm + h->offsets[cb], h->d_ctr, &h->parity, h->hrt_done, &h->hrt_pending, false};
    return run_host_roundtrip(h, b, step0, T, cb, ce, stream, sc);
}

}  // namespace

extern "C" {

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
    if (prop.multiProcessorCount < 1 || prop.maxSharedMemoryPerMultiProcessor < 64u * 1024u) return RC_E_DEVICE;

    rc_cohort* h = new (std::nothrow) rc_cohort();
    if (!h) return RC_E_NOMEM;
    DeviceGuard guard(hip_device);
    if (!guard.ok) { delete h; return RC_E_DEVICE; }
    h->device = hip_device;
    h->n_cu = (uint32_t)prop.multiProcessorCount;
    h->lds_per_cu = prop.maxSharedMemoryPerMultiProcessor;
    // the full mask image up to 45% of a CU's LDS (72 KB of 160 KB); two
    // workgroups per CU below half of it
    const size_t full_image_limit = h->lds_per_cu * 9u / 20u;
    const size_t lds_two_per_cu = h->lds_per_cu / 2u;
    h->N = desc->n_sessions;
    h->W = desc->n_words;
    h->R = desc->n_routes;
    h->C = desc->n_cohorts;
    h->thr = desc->decide_thr;
    h->wmax = next_pow2_words(h->W);
    h->exact = (h->wmax == h->W);
    const uint32_t R = h->R;
    // with a single route both route maps give route 0
    h->ra.mode = (desc->route_mode == RC_ROUTE_CDF && R > 1u) ? RC_ROUTE_CDF : RC_ROUTE_MOD;
    h->ra.n_routes = R;
    h->ra.is_pow2 = (R & (R - 1u)) == 0u;
    h->ra.pow2_mask = h->ra.is_pow2 ? R - 1u : 0u;
    h->ra.cdf_n = (h->ra.mode == RC_ROUTE_CDF) ? R - 1u : 0u;
    h->route_kind = h->ra.mode == RC_ROUTE_CDF ? RK_CDF : (h->ra.is_pow2 ? RK_POW2 : RK_MOD);
    h->ra.cdf_top = 0;
    while (h->ra.cdf_n && (h->ra.cdf_top << 1) <= h->ra.cdf_n && h->ra.cdf_top < (1u << 30))
        h->ra.cdf_top = h->ra.cdf_top ? h->ra.cdf_top << 1 : 1u;

    // table image layout (see the file comment)
    const size_t full_bytes = (size_t)(R + 1u) * (h->wmax + 4u) * 4u;
    h->full = h->wmax <= 16u || full_bytes <= full_image_limit;
    // Full image: [word-0 masks | CDF thresholds | guide] (the chain
    // section, everything the word-0 chain reads), then the mask rows, then
    // the tool pairs.  Table image: the raw rows, then thresholds and guide.
    const uint32_t row_words = h->full ? h->wmax : 16u;
    const uint32_t tab_words = (R + 1u) * (h->full ? row_words + 4u : row_words);
    auto pad4 = [](uint32_t x) { return (x + 3u) & ~3u; };
    const uint32_t m0_words = h->full ? pad4(R + 1u) : 0u;
    h->cdf_off = h->full ? m0_words : tab_words;
    h->guide_off = h->cdf_off + pad4(h->ra.cdf_n);
    const uint32_t after_guide = h->full ? tab_words + pad4(R) : 0u;  // rows and tools
    // The chain kernel's LDS after the image: the count exchange ([16][nwave +
    // 4] words; the table chain uses the first [2][nwave + 4]), then (full
    // image, WMAX >= 16: the two-role or the pipelined split) the control
    // handed to the replaying lanes, 16 steps of a 4-byte addend and a 4-byte
    // control word per lane, then (full image) the effect stage of
    // sub-wavefront bins, 4 + 16 bytes per lane.
    h->nwave = h->full ? 4u : 8u;
    const bool ctl_area = h->full && h->wmax >= 16u;
    const uint32_t na = h->nwave * 64u;
    const size_t lds_after_image = 16u * (h->nwave + 4u) * 4u + (ctl_area ? 16u * na * 8u : 0u) +
                                   (h->full ? na * 20u : 0u);
    uint32_t guide_bits = 0, guide_n = 0;
    if (h->ra.mode == RC_ROUTE_CDF) {
        // Eight buckets per route, at most 2^12: with skewed routes the
        // thresholds of the light routes crowd into few buckets, and every
        // threshold in a bucket is a dependent LDS step of the chain's search
        // (Zipf(1.1) over 64 routes: at most 1 per bucket, 2 with four
        // buckets per route).  Fewer buckets when that keeps two workgroups
        // on a CU that the smallest guide would allow.
        const uint32_t gmin = ceil_log2(R) < 1u ? 1u : ceil_log2(R);
        guide_bits = gmin + 3u < 12u ? gmin + 3u : (gmin > 12u ? gmin : 12u);
        auto lds_at = [&](uint32_t gb) {
            return ((size_t)h->guide_off + pad4((1u << gb) + 1u) + after_guide) * 4u + lds_after_image;
        };
        if (lds_at(gmin) <= lds_two_per_cu)
            while (guide_bits > gmin && lds_at(guide_bits) > lds_two_per_cu) --guide_bits;
        guide_n = (1u << guide_bits) + 1u;
        h->ra.guide_shift = 32u - guide_bits;
    }
    const uint32_t guide_end = h->guide_off + pad4(guide_n);
    h->chain_words = h->full ? guide_end : 0u;
    h->rows_off = h->full ? guide_end : 0u;
    h->tools_off = h->rows_off + tab_words;
    h->img_words = h->full ? h->tools_off + pad4(R) : guide_end;
    const size_t lds_image = (size_t)h->img_words * 4u;
    // chain_threads is the two-role (W >= 32) or one-lane workgroup; the
    // pipelined split launches three lanes per session.
    const bool split = h->full && h->wmax >= 32u;
    h->chain_threads = (split ? 2u : 1u) * na;
    h->chain_lds_bytes = lds_image + lds_after_image;

    h->offsets.assign(desc->cohort_offsets, desc->cohort_offsets + h->C + 1u);
    build_plan(h->offsets.data(), h->C, h->nwave, h->plan);

    int rc = RC_OK;
    if (rc == RC_OK) rc = dev_upload(&h->d_offsets, h->offsets.data(), h->offsets.size() * 4u);
    if (rc == RC_OK) rc = dev_upload(&h->d_raw, desc->table, (size_t)R * 16u * 4u);
    if (rc == RC_OK) rc = dev_upload(&h->d_cdf, desc->route_cdf, (size_t)h->ra.cdf_n * 4u);
    if (rc == RC_OK && hipMalloc((void**)&h->d_img, (size_t)h->img_words * 4u) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMalloc((void**)&h->d_span, 16) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMemset(h->d_span, 0, 16) != hipSuccess) rc = RC_E_DEVICE;
    if (rc == RC_OK) rc = dev_upload(&h->d_wdesc, h->plan.wdesc.data(), h->plan.wdesc.size() * 4u);
    if (rc == RC_OK && hipMalloc((void**)&h->d_perm, (size_t)h->N * sizeof(uint32_t)) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMalloc((void**)&h->d_ctr, 2 * sizeof(uint32_t)) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipMemset(h->d_ctr, 0, 2 * sizeof(uint32_t)) != hipSuccess) rc = RC_E_DEVICE;
    if (rc == RC_OK && hipHostMalloc((void**)&h->h_word, sizeof(uint32_t), hipHostMallocDefault) != hipSuccess) rc = RC_E_NOMEM;
    if (rc == RC_OK && hipEventCreateWithFlags(&h->hrt_done, hipEventDisableTiming) != hipSuccess) rc = RC_E_DEVICE;
    if (rc == RC_OK) rc = noalloc_init(hip_device);
    if (rc == RC_OK) {
        ImageArgs ia;
        ia.raw = h->d_raw;
        ia.cdf = h->d_cdf;
        ia.img = h->d_img;
        ia.max_span = h->d_span;
        ia.n_routes = R;
        ia.row_words = row_words;
        ia.full = h->full ? 1u : 0u;
        ia.tab_words = tab_words;
        ia.tools_off = h->tools_off;
        ia.cdf_off = h->cdf_off;
        ia.cdf_n = h->ra.cdf_n;
        ia.guide_off = h->guide_off;
        ia.guide_n = guide_n;
        ia.guide_shift = h->ra.guide_shift;
        ia.total_words = h->img_words;
        ia.m0_words = m0_words;
        ia.rows_off = h->rows_off;
        hipLaunchKernelGGL(rc_prep_kernel, dim3((h->img_words + 255u) / 256u), dim3(256), 0, 0, ia);
        uint32_t span = 0;
        if (launch_ok() != RC_OK || hipMemcpy(&span, h->d_span, 4, hipMemcpyDeviceToHost) != hipSuccess)
            rc = RC_E_DEVICE;
        h->ra.guide_top = 0;
        while (span && (h->ra.guide_top << 1) <= span) h->ra.guide_top = h->ra.guide_top ? h->ra.guide_top << 1 : 1u;
    }
    for (int v = 0; v < 4 && rc == RC_OK; ++v) {
        const bool fl = (v & 1) != 0, piped = (v & 2) != 0;
        if (piped && !has_piped(h->wmax, h->full)) continue;
        ChainFn fn = pick_chain(h->wmax, h->exact, h->full, piped, h->route_kind, fl);
        if (!fn) rc = RC_E_DEVICE;
        if (rc == RC_OK && hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)h->chain_lds_bytes) != hipSuccess) rc = RC_E_DEVICE;
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
    return run_host_roundtrip_handle(h, b, step0, n_steps, cohort_begin, cohort_end, stream);
}

int rc_cohort_run_chain_noalloc(rc_cohort* h, const rc_buffers* b, uint32_t step0, uint32_t n_steps,
                                int mode, uint32_t cohort_begin, uint32_t cohort_end, void* hip_stream) {
    if (!h || !b) return RC_E_INVALID;
    if (mode != RC_MODE_RESIDENT && mode != RC_MODE_HOST_ROUNDTRIP) return RC_E_INVALID;
    if (cohort_begin > cohort_end || cohort_end > h->C) return RC_E_INVALID;
    if (h->offsets[cohort_end] - h->offsets[cohort_begin] > RC_NOALLOC_MAX_SESSIONS) return RC_E_INVALID;
    DeviceGuard guard(h->device);
    if (!guard.ok) return RC_E_DEVICE;
    const int v = validate_buffers(h, b, n_steps);
    if (v != RC_OK) return v;
    h->last_launches = 0;
    h->last_d2h = 0;
    if (n_steps == 0u || cohort_begin == cohort_end) return RC_OK;
    hipStream_t stream = (hipStream_t)hip_stream;
    // the resident chain uses no scratch
    if (mode == RC_MODE_RESIDENT) return run_resident(h, b, step0, n_steps, cohort_begin, cohort_end, stream);
    uint32_t* base = g_noalloc_ptr[h->device];  // resolved by rc_cohort_create
    if (!base) return RC_E_DEVICE;
    uint32_t parity = 0;
    HrtScratch sc{base + NOALLOC_PERM_OFF, base, &parity, g_noalloc_done[h->device],
                  &g_noalloc_pending[h->device], true};
    return run_host_roundtrip(h, b, step0, n_steps, cohort_begin, cohort_end, stream, sc);
}

int rc_cohort_run_floor(rc_cohort* h, const rc_buffers* b, const uint32_t* decisions, uint32_t n_steps,
                        uint32_t cohort_begin, uint32_t cohort_end, void* hip_stream) {
    if (!h || !b || !decisions) return RC_E_INVALID;
    if (cohort_begin > cohort_end || cohort_end > h->C) return RC_E_INVALID;
    DeviceGuard guard(h->device);
    if (!guard.ok) return RC_E_DEVICE;
    const int v = validate_buffers(h, b, n_steps, true, decisions);
    if (v != RC_OK) return v;
    h->last_launches = 0;
    h->last_d2h = 0;
    if (n_steps == 0u || cohort_begin == cohort_end) return RC_OK;
    return run_resident(h, b, 0u, n_steps, cohort_begin, cohort_end, (hipStream_t)hip_stream, decisions);
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
    if (n_workgroups) *n_workgroups = h->plan.n_bins;
    if (lanes_per_workgroup) *lanes_per_workgroup = h->nwave * 64u;
    if (idle_lanes) *idle_lanes = h->plan.idle_lanes;
    return RC_OK;
}

}  // extern "C"
