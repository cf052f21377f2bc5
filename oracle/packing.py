"""Oracle of the cohort shares: fixed-partition eligibility F, the exact
offline packing P* with a witness schedule, and the local-overlap bound U.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  Plain Python
integers, written from the definitions, for the test sizes; nothing here is
blocked, fused or reordered beyond what the definitions state.

Model (Section 3 "Events and the hardware threshold" and "Four shares"):
event i has an integer-nanosecond release t_i, a latest launch d_i = t_i +
delta (the equal relative deadlines of Section 4) and a route r_i.  A batch
(tau, B) is feasible when |B| >= K_r, every member has route r, and
t_i <= tau <= d_i for every member (Eq. feasible-batch).  Comparisons are
inclusive, on the integer clock (Section 4 "Exact clock").

* F (Eq. fixed): windows [w0 + k delta, w0 + (k+1) delta) (origin-aligned,
  half-open, Section 5 "Stationary replay"); a bucket is (window, route) and
  counts when it holds at least K_r events.
* P* (Eq. dp, Section 4): per route, releases sorted ascending,
  D[0] = 0 and D[j] = max(D[j-1], max over starts i with i <= j-K+1 and
  t_j - t_i <= delta of D[i-1] + j - i + 1); the witness follows the
  back-pointers from D[n].
* U (Eq. upper): event i counts when the active same-route count
  Q_r(tau) = #{j : r_j = r, t_j <= tau <= d_j} reaches K_r at some tau in
  [t_i, d_i].
* A subset brute force over every feasible schedule, for tiny inputs.
All functions return event counts (numerators); shares divide by |E|.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple


def _k(k, r) -> int:
    return int(k[r]) if isinstance(k, (list, tuple, dict)) else int(k)


def _by_route(t: Sequence[int], r: Sequence[int]) -> Dict[int, List[Tuple[int, int]]]:
    """route -> [(release, event index)] in ascending release (ties by index)."""
    out: Dict[int, List[Tuple[int, int]]] = {}
    for i, (ti, ri) in enumerate(zip(t, r)):
        out.setdefault(int(ri), []).append((int(ti), i))
    for v in out.values():
        v.sort()
    return out


def fixed_eligible(t, r, K, delta: int, origin: int = 0) -> int:
    """Numerator of F: events in (window, route) buckets of at least K_r."""
    buckets: Dict[Tuple[int, int], int] = {}
    for ti, ri in zip(t, r):
        w = (int(ti) - origin) // delta  # floor division: half-open windows
        buckets[(w, int(ri))] = buckets.get((w, int(ri)), 0) + 1
    return sum(n for (w, rr), n in buckets.items() if n >= _k(K, rr))


def exact_packing(t, r, K, delta: int):
    """Numerator of P* and a witness: a list of batches, each a list of event
    indices (one route, at least K_r events, release span at most delta)."""
    total = 0
    witness: List[List[int]] = []
    for rr, ev in sorted(_by_route(t, r).items()):
        k = _k(K, rr)
        n = len(ev)
        ts = [x[0] for x in ev]  # ts[j - 1] is t_j of the 1-based recurrence
        D = [0] * (n + 1)
        back = [0] * (n + 1)  # 0: event j unassigned; else the block's start i
        for j in range(1, n + 1):
            D[j] = D[j - 1]
            back[j] = 0
            for i in range(1, j - k + 2):  # i <= j - K + 1
                if ts[j - 1] - ts[i - 1] <= delta:
                    cand = D[i - 1] + j - i + 1
                    if cand > D[j]:
                        D[j] = cand
                        back[j] = i
        total += D[n]
        j = n
        while j > 0:
            i = back[j]
            if i == 0:
                j -= 1
            else:
                witness.append([ev[m - 1][1] for m in range(i, j + 1)])
                j = i - 1
    return total, witness


def local_overlap(t, r, K, delta: int) -> int:
    """Numerator of U.  Q_r is a step function that only rises at releases, so
    its maximum over [t_i, d_i] is attained at t_i or at a same-route release
    inside that interval; each candidate is counted directly."""
    count = 0
    groups = _by_route(t, r)
    for ti, ri in zip(t, r):
        ti, ri = int(ti), int(ri)
        same = [x[0] for x in groups[ri]]
        cands = [ti] + [tj for tj in same if ti <= tj <= ti + delta]
        best = max(sum(1 for tj in same if tj <= tau <= tj + delta) for tau in cands)
        if best >= _k(K, ri):
            count += 1
    return count


def batch_is_feasible(batch: Sequence[int], t, r, K, delta: int) -> bool:
    """Eq. feasible-batch for a batch of event indices: one route, at least K
    members, and a launch time inside every member's [t_i, t_i + delta]
    (which exists exactly when max t <= min t + delta)."""
    if not batch:
        return False
    routes = {int(r[i]) for i in batch}
    if len(routes) != 1 or len(set(batch)) != len(batch):
        return False
    rr = routes.pop()
    ts = [int(t[i]) for i in batch]
    return len(batch) >= _k(K, rr) and max(ts) <= min(ts) + delta


def brute_force_packing(t, r, K, delta: int) -> int:
    """Maximum number of events covered by disjoint feasible batches, by
    exhaustive search over assignments (tiny inputs only)."""
    n = len(t)
    best = 0

    def rec(idx: int, batches: List[List[int]], assigned: int):
        nonlocal best
        if idx == n:
            if all(batch_is_feasible(b, t, r, K, delta) for b in batches):
                best = max(best, assigned)
            return
        # bound: even assigning every remaining event cannot beat best
        if assigned + (n - idx) <= best:
            return
        rec(idx + 1, batches, assigned)  # leave event idx unassigned
        for b in batches:  # join an open batch
            b.append(idx)
            rec(idx + 1, batches, assigned + 1)
            b.pop()
        batches.append([idx])  # open a new batch
        rec(idx + 1, batches, assigned + 1)
        batches.pop()

    rec(0, [], 0)
    return best


def shares(t, r, K, delta: int, origin: int = 0):
    """(F, P*, U) numerators and the witness."""
    f = fixed_eligible(t, r, K, delta, origin)
    p, w = exact_packing(t, r, K, delta)
    u = local_overlap(t, r, K, delta)
    return f, p, u, w
