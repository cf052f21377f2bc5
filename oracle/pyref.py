"""Second, independent formulation of the transition with Python integers.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  It is written from the
same definition as the C oracle but shares none of its code: arithmetic is on
unbounded Python ints reduced modulo 2^32, the rotation is the closed form
(x * 2^k mod 2^32) + floor(x / 2^(32 - k)), and the compaction is Python's
``sorted`` with the key (not taken, session id), a textbook stable partition.
It is slow and meant for tiny inputs only.

Paper passages: the unit of work (Abstract; Section 2 "Unit of execution"),
the predicate and the two route bodies (Section 7 "Matched mechanisms"), the
per-event compaction and effect ordering (Section 11 "Mechanism and sampling
scope").
"""
from __future__ import annotations

MOD32 = 1 << 32


def fmix32(h: int) -> int:
    """MurmurHash3 32-bit finalizer (A. Appleby, public domain)."""
    h %= MOD32
    h ^= h >> 16
    h = (h * 0x85EBCA6B) % MOD32
    h ^= h >> 13
    h = (h * 0xC2B2AE35) % MOD32
    h ^= h >> 16
    return h


def rotl(x: int, k: int) -> int:
    """Rotation left by k mod 32, as (x * 2^k mod 2^32) + floor(x / 2^(32-k))."""
    k %= 32
    if k == 0:
        return x % MOD32
    return (x * (1 << k)) % MOD32 + x // (1 << (32 - k))


def route(o: int, n_routes: int, route_mode: int, cdf=()) -> int:
    if route_mode == 0:
        return o % n_routes
    return sum(1 for v in cdf if int(v) <= o)


def session_step(words, o, step, n_routes, table, route_mode, cdf, thr, forced=None):
    """One session's transition: returns (new_words, taken, route, tool).

    ``forced``: None, or the decision to use instead of the predicate (the
    no-decision floor replays a recorded decision sequence)."""
    r = route(o, n_routes, route_mode, cdf)
    if forced is None:
        taken = (fmix32(words[0] ^ o ^ (step % MOD32)) % 65536) < thr
    else:
        taken = bool(forced)
    if taken:
        new = [x ^ ((int(table[r][w % 16]) * (w + 1)) % MOD32)
               for w, x in enumerate(words)]
    else:
        new = [(rotl(x, r + 1) + o) % MOD32 for x in words]
    tool = int(table[r][1 if taken else 0]) % 8
    return new, taken, r, tool


def run_chain(sessions, outcomes, cohorts, n_steps, step0, n_routes, table,
              route_mode, cdf, thr, forced=None):
    """Chained steps over a list of cohorts.

    ``sessions``: dict sid -> list of W words; ``outcomes``: dict sid -> int;
    ``cohorts``: list of lists of sids (each in ascending order).
    ``forced``: None, or a function (t, sid) -> decision replacing the
    predicate (the no-decision floor).
    Returns (sessions, outcomes, effects, counts) where ``effects[t][c]`` is
    the list of (sid, tool, payload tuple) in emitted order and
    ``counts[t][c]`` the taken count.
    """
    sessions = {s: list(v) for s, v in sessions.items()}
    outcomes = dict(outcomes)
    effects, counts = [], []
    for t in range(n_steps):
        step = (step0 + t) % MOD32
        eff_t, cnt_t = [], []
        for members in cohorts:
            results = {}
            for s in members:
                results[s] = session_step(sessions[s], outcomes[s], step,
                                          n_routes, table, route_mode, cdf, thr,
                                          None if forced is None else forced(t, s))
            order = sorted(members, key=lambda s: (not results[s][1], s))
            eff_t.append([(s, results[s][3], tuple(results[s][0][:4])) for s in order])
            cnt_t.append(sum(1 for s in members if results[s][1]))
            for s in members:
                sessions[s] = results[s][0]
                outcomes[s] = fmix32(sessions[s][0])
        effects.append(eff_t)
        counts.append(cnt_t)
    return sessions, outcomes, effects, counts
