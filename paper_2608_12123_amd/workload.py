"""Seeded synthetic inputs for the ready-cohort transition.

This module only *generates inputs*: it holds none of the transition's
arithmetic (no routing, decision, update, compaction or chaining).  Both the
HIP path and the oracle consume what it produces, which is the only thing
they share.

* Random words come from SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014), one counter-based stream per
  (workload, chunk, array), keyed from the root seed 20260811 (the replay root
  seed of the paper's Section 5 grid).  A uint32 draw is the high half of a
  64-bit output.
* Route keys follow the outcome-derived route key of Section 5 ("Trace
  source"/route-key grouping).  For Zipf-distributed route keys the route map
  is a threshold table ("CDF mode"): route k owns the outcomes in
  [cdf[k-1], cdf[k]).  The thresholds are derived from the Zipf law in double
  precision here and handed to both sides as data.
* The 1M-session workload forms variable cohorts from Poisson arrivals with a
  50 ms launch deadline (the arrival model of Section 5 "Stationary replay"
  and the primary 50 ms deadline), floored to K in {32, 64, 128, 256} (the K
  grid of Section 5), on an integer-nanosecond clock (Section 4 "Exact
  clock").  It is synthetic: no trace record is used.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

ROOT_SEED = 20260811
GAMMA = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1

ROUTE_MOD = 0
ROUTE_CDF = 1

# array identifiers for stream keys
A_STATE, A_OUTCOME, A_TABLE, A_ARRIVAL, A_ARRIVAL_OUTCOME = 1, 2, 3, 4, 5


# --------------------------------------------------------------------------
# SplitMix64
# --------------------------------------------------------------------------
def _mix64_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def _mix64(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def splitmix64(seed: int, n: int, start: int = 0) -> np.ndarray:
    """Outputs start..start+n-1 of the SplitMix64 sequence seeded with ``seed``."""
    idx = np.arange(start + 1, start + n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & MASK64) + idx * np.uint64(GAMMA)
    return _mix64(z)


def stream_seed(*keys: int, root: int = ROOT_SEED) -> int:
    """Seed of the stream identified by ``keys`` under ``root``."""
    x = root & MASK64
    for k in keys:
        x = _mix64_int(x + GAMMA * ((k & MASK64) + 1))
    return x


def uniform_u32(n: int, *keys: int, root: int = ROOT_SEED, start: int = 0) -> np.ndarray:
    """``n`` uniform uint32 values of the stream ``keys`` (high 32 bits)."""
    seed = stream_seed(*keys, root=root)
    out = np.empty(n, dtype=np.uint32)
    step = 1 << 20
    for a in range(0, n, step):
        b = min(n, a + step)
        out[a:b] = splitmix64(seed, b - a, start + a) >> np.uint64(32)
    return out


def uniform_unit(n: int, *keys: int, root: int = ROOT_SEED) -> np.ndarray:
    """``n`` doubles in [0, 1) from the top 53 bits of the stream ``keys``."""
    z = splitmix64(stream_seed(*keys, root=root), n)
    return (z >> np.uint64(11)).astype(np.float64) * (1.0 / (1 << 53))


def device_uniform_u32(shape, *keys: int, device, root: int = ROOT_SEED):
    """Uniform uint32 values, as int32 bit patterns, drawn on a torch device
    by torch's seeded generator for that device (keyed like the host
    streams).  For inputs too large to draw on the host; a test that checks
    them copies the slices it needs to the host before they are used."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(stream_seed(*keys, root=root) & ((1 << 63) - 1))
    return torch.randint(-(1 << 31), 1 << 31, tuple(shape), dtype=torch.int32, device=device,
                         generator=g)


# --------------------------------------------------------------------------
# Derived route data and thresholds
# --------------------------------------------------------------------------
def threshold_from_p(p: float) -> int:
    """Integer decision threshold for a taken probability p: round-half-up of
    p * 65536 (p = 0.5 gives 32768, 0.3 gives 19661, 0.05 gives 3277)."""
    return int(math.floor(p * 65536.0 + 0.5))


def zipf_cdf(n_routes: int, s: float) -> np.ndarray:
    """R-1 nondecreasing uint32 thresholds of a Zipf(s) route law.

    cdf[k] = floor(2^32 * sum_{j<=k} (j+1)^-s / sum_{j<R} (j+1)^-s), k < R-1;
    rank 1 is route 0.
    """
    w = np.arange(1, n_routes + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w) / np.sum(w)
    th = np.floor(c[:-1] * 4294967296.0)
    return np.minimum(th, 4294967295.0).astype(np.uint32)


def route_of_outcomes_cdf(outcomes: np.ndarray, cdf: np.ndarray) -> np.ndarray:
    """Route keys of step-0 outcomes under a threshold table, used only to
    group arrivals into cohorts (numpy's searchsorted; the transition's own
    route step is implemented independently by each side)."""
    return np.searchsorted(cdf, outcomes, side="right").astype(np.int64)


def uniform_offsets(n_sessions: int, k: int) -> np.ndarray:
    """Cohort offsets for cohorts of size k, the last one partial."""
    b = list(range(0, n_sessions, k)) + [n_sessions]
    return np.asarray(b, dtype=np.uint32)


# --------------------------------------------------------------------------
# Cohort former for variable cohorts (deadline-or-full, per route)
# --------------------------------------------------------------------------
def poisson_arrivals_ns(n: int, rate_per_s: float, *keys: int) -> np.ndarray:
    """Integer-ns arrival times of a homogeneous Poisson process."""
    u = uniform_unit(n, *keys)
    gaps = -np.log1p(-u) / rate_per_s
    return np.round(np.cumsum(gaps) * 1e9).astype(np.int64)


def form_cohorts(times_ns: np.ndarray, routes: np.ndarray, deadline_ns: int,
                 sizes=(32, 64, 128, 256)) -> Tuple[np.ndarray, Dict[str, int]]:
    """Deadline-or-full cohort former.

    For each route, in release order: a cohort opens at the first waiting
    arrival and closes at the earlier of its max(sizes)-th arrival or
    open + deadline (inclusive).  Its size is floored to the largest allowed
    size not above the arrivals it holds; the rest stay waiting.  With fewer
    than min(sizes) arrivals at the deadline it waits for the min(sizes)-th
    arrival ("late").  A route's final remainder below min(sizes) forms one
    partial cohort.

    Returns (order, stats): ``order`` lists arrival indices grouped into
    cohorts, cohorts sorted by (close time, route); and the cohort sizes in
    ``stats['sizes']`` (as an array under key 'sizes_array').
    """
    ks = sorted(sizes)
    kmin, kmax = ks[0], ks[-1]
    cohorts: List[Tuple[int, int, np.ndarray]] = []  # (close_ns, route, idx)
    late = 0
    order_all = np.argsort(routes, kind="stable")
    r_sorted = routes[order_all]
    bounds = np.searchsorted(r_sorted, np.arange(int(routes.max()) + 2))
    for r in range(int(routes.max()) + 1):
        idx = order_all[bounds[r]:bounds[r + 1]]
        if idx.size == 0:
            continue
        t = times_ns[idx]  # already increasing: stable sort of increasing times
        n = idx.size
        i = 0
        while i < n:
            left = n - i
            m = int(np.searchsorted(t, t[i] + deadline_ns, side="right")) - i
            m = min(m, kmax)
            if m >= kmin:
                k = max(s for s in ks if s <= m)
                close = int(t[i + kmax - 1]) if m >= kmax else int(t[i] + deadline_ns)
            elif left >= kmin:
                k = kmin
                close = int(t[i + kmin - 1])
                late += 1
            else:
                k = left
                close = int(t[-1])
            cohorts.append((close, r, idx[i:i + k]))
            i += k
    cohorts.sort(key=lambda x: (x[0], x[1]))
    order = np.concatenate([c[2] for c in cohorts])
    sizes_arr = np.asarray([c[2].size for c in cohorts], dtype=np.int64)
    stats = {"n_cohorts": len(cohorts), "late": late}
    for k in ks:
        stats["k%d" % k] = int(np.sum(sizes_arr == k))
    stats["partial"] = int(np.sum(~np.isin(sizes_arr, ks)))
    return order, {"stats": stats, "sizes_array": sizes_arr}


# --------------------------------------------------------------------------
# The five benchmark workloads
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    key: str              # short name
    cid: int              # stream key of the workload
    title: str
    n_words: int          # W
    n_routes: int         # R
    route_mode: int       # ROUTE_MOD or ROUTE_CDF
    zipf_s: float         # Zipf exponent (CDF mode)
    decide_thr: int       # integer threshold
    n_steps: int          # T
    cohort_size: int      # K for uniform cohorts; 0 = variable (former)
    n_sessions: int       # sessions per descriptor (chunk)
    invocations: int      # independent invocations (1 = one launch over all)
    per_cohort_invocation: bool  # an invocation is one cohort range


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, "B=32 sessions, W=8, R=4 mod, p=0.5, T=1, 1000 invocations",
                     8, 4, ROUTE_MOD, 0.0, threshold_from_p(0.5), 1, 32, 32 * 1000, 1000, True),
    "k64": Workload("k64", 2, "cohort K=64, W=16, R=16 mod, p=0.5, T=8, 10000 invocations",
                    16, 16, ROUTE_MOD, 0.0, threshold_from_p(0.5), 8, 64, 64 * 1000, 10000, True),
    "k256": Workload("k256", 3, "cohort K=256, W=32, R=64 Zipf(1.1), p=0.3, T=32, 50000 invocations",
                     32, 64, ROUTE_CDF, 1.1, threshold_from_p(0.3), 32, 256, 256 * 1000, 50000, True),
    "s100k": Workload("s100k", 4, "100,000 sessions in 391 cohorts of K=256, W=32, R=256 mod, p=0.5, T=16",
                      32, 256, ROUTE_MOD, 0.0, threshold_from_p(0.5), 16, 256, 100000, 1, False),
    "s1m": Workload("s1m", 5, "1,000,000 sessions, variable cohorts K in {32,64,128,256}, W=64, "
                    "R=1024 Zipf(1.1), p=0.05, T=16",
                    64, 1024, ROUTE_CDF, 1.1, threshold_from_p(0.05), 16, 0, 1000000, 1, False),
}
WORKLOAD_ORDER = ["tiny", "k64", "k256", "s100k", "s1m"]

ARRIVAL_RATE_PER_S = 2.0e5     # mean 10,000 arrivals per 50 ms window
DEADLINE_NS = 50_000_000


@dataclasses.dataclass
class Inputs:
    """One descriptor's worth of inputs (host numpy arrays)."""
    workload: Workload
    chunk: int
    n_sessions: int
    n_words: int
    n_routes: int
    route_mode: int
    decide_thr: int
    n_steps: int
    cohort_offsets: np.ndarray   # uint32 [C+1]
    table: np.ndarray            # uint32 [R][16]
    route_cdf: Optional[np.ndarray]  # uint32 [R-1] or None
    state: np.ndarray            # uint32 [W][ld]
    outcome: np.ndarray          # uint32 [ld]
    former_stats: Optional[dict] = None

    @property
    def n_cohorts(self) -> int:
        return int(self.cohort_offsets.size - 1)

    @property
    def ld(self) -> int:
        return int(self.state.shape[1])

    def copy_state(self):
        return self.state.copy(), self.outcome.copy()


def n_chunks(wl: Workload) -> int:
    if not wl.per_cohort_invocation:
        return 1
    per_chunk = wl.n_sessions // wl.cohort_size
    return (wl.invocations + per_chunk - 1) // per_chunk


def make_inputs(wl: Workload, chunk: int = 0, ld: Optional[int] = None,
                root: int = ROOT_SEED) -> Inputs:
    """Generate the inputs of chunk ``chunk`` of workload ``wl``.

    Uniform workloads: cohorts of ``cohort_size`` (the last one partial).
    The variable workload: cohorts from :func:`form_cohorts`; sessions are
    numbered in cohort order and each session's step-0 outcome is its
    arrival's outcome.
    """
    R, W = wl.n_routes, wl.n_words
    table = uniform_u32(R * 16, wl.cid, A_TABLE, root=root).reshape(R, 16)
    cdf = zipf_cdf(R, wl.zipf_s) if wl.route_mode == ROUTE_CDF else None
    stats = None
    if wl.cohort_size:
        N = wl.n_sessions
        offsets = uniform_offsets(N, wl.cohort_size)
        outcome0 = uniform_u32(N, wl.cid, chunk, A_OUTCOME, root=root)
    else:
        N = wl.n_sessions
        times, routes, arr_out = arrival_events(wl, chunk, root=root)
        order, info = form_cohorts(times, routes, DEADLINE_NS)
        outcome0 = arr_out[order]
        offsets = np.concatenate([[0], np.cumsum(info["sizes_array"])]).astype(np.uint32)
        stats = info["stats"]
    ld = N if ld is None else ld
    assert ld >= N
    state = np.zeros((W, ld), dtype=np.uint32)
    state[:, :N] = uniform_u32(W * N, wl.cid, chunk, A_STATE, root=root).reshape(W, N)
    outcome = np.zeros(ld, dtype=np.uint32)
    outcome[:N] = outcome0
    if ld > N:  # poison the padding columns so untouched-region checks mean something
        state[:, N:] = 0xA5A5A5A5
        outcome[N:] = 0x5A5A5A5A
    return Inputs(wl, chunk, N, W, R, wl.route_mode, wl.decide_thr, wl.n_steps,
                  offsets, table, cdf, state, outcome, stats)


def arrival_events(wl: Workload, chunk: int = 0, root: int = ROOT_SEED):
    """The control events of a variable-cohort workload: integer-ns Poisson
    releases, the route of each arrival (of its outcome, by the workload's
    route rule) and the arrival outcomes.  Returns (times, routes, outcomes)."""
    assert not wl.cohort_size, "uniform workloads have no arrival stream"
    N, R = wl.n_sessions, wl.n_routes
    times = poisson_arrivals_ns(N, ARRIVAL_RATE_PER_S, wl.cid, chunk, A_ARRIVAL)
    arr_out = uniform_u32(N, wl.cid, chunk, A_ARRIVAL_OUTCOME, root=root)
    if wl.route_mode == ROUTE_CDF:
        routes = route_of_outcomes_cdf(arr_out, zipf_cdf(R, wl.zipf_s))
    else:
        routes = arr_out % R
    return times, routes.astype(np.uint32), arr_out


def make_custom(*, n_words: int, n_routes: int, route_mode: int, decide_thr: int,
                cohort_sizes, n_steps: int, zipf_s: float = 1.1, seed_key: int = 0,
                ld: Optional[int] = None, table: Optional[np.ndarray] = None,
                route_cdf: Optional[np.ndarray] = None) -> Inputs:
    """Inputs of an arbitrary shape (tests): cohorts of the given sizes."""
    sizes = np.asarray(list(cohort_sizes), dtype=np.int64)
    assert sizes.size >= 1 and np.all(sizes >= 1)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    N = int(offsets[-1])
    key = 1000 + (seed_key & 0xFFFFFF)
    if table is None:
        table = uniform_u32(n_routes * 16, key, A_TABLE).reshape(n_routes, 16)
    if route_mode == ROUTE_CDF and route_cdf is None:
        route_cdf = zipf_cdf(n_routes, zipf_s)
    wl = Workload("custom", key, "custom", n_words, n_routes, route_mode, zipf_s,
                  decide_thr, n_steps, 0, N, 1, False)
    ld = N if ld is None else ld
    state = np.zeros((n_words, ld), dtype=np.uint32)
    state[:, :N] = uniform_u32(n_words * N, key, 0, A_STATE).reshape(n_words, N)
    outcome = np.zeros(ld, dtype=np.uint32)
    outcome[:N] = uniform_u32(N, key, 0, A_OUTCOME)
    if ld > N:
        state[:, N:] = 0xA5A5A5A5
        outcome[N:] = 0x5A5A5A5A
    return Inputs(wl, 0, N, n_words, n_routes, route_mode, decide_thr, n_steps,
                  offsets, np.ascontiguousarray(table, dtype=np.uint32),
                  None if route_cdf is None else np.ascontiguousarray(route_cdf, dtype=np.uint32),
                  state, outcome, None)


def transitions_per_invocation(inp: Inputs, wl: Workload) -> int:
    if wl.per_cohort_invocation:
        return wl.cohort_size * wl.n_steps
    return inp.n_sessions * wl.n_steps
