"""Pins of the oracle to facts other than its own code.

Each ``pin_*`` function takes an :class:`oracle.Oracle` and raises
``AssertionError`` when the oracle disagrees with a fact fixed by the
mathematics or by a published reference:

* published MurmurHash3_x86_32 verification vectors (tests/golden/);
* closed forms of rotation, of the two route bodies in special cases
  (all-ones / single-column tables, rotation period, XOR involution);
* the exact decision rate over all 2^32 outcomes (fmix32 is a bijection, so
  exactly thr * 65536 outcomes are taken);
* exact route histograms against interval lengths;
* textbook routines for the compaction (Python's stable ``sorted``);
* invariants of the chain (effect count, per-cohort counts, next outcome,
  untouched regions, composability of chains);
* a brute-force cross-check on tiny domains against the second, independent
  Python formulation.

The functions are shared by ``test_oracle_pins.py`` (the real oracle must
pass every pin) and ``test_oracle_mutants.py`` (a deliberately broken oracle
must fail at least one).
"""
from __future__ import annotations

import itertools
import math
import os

import numpy as np

from oracle import ROUTE_CDF, ROUTE_MOD, pyref

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
M32 = (1 << 32) - 1
SPECIAL = [0, 1, 2, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFE, 0xFFFFFFFF, 0x12345678, 0xDEADBEEF]


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------
def murmur3_x86_32(oracle, key: bytes, seed: int) -> int:
    """MurmurHash3_x86_32 body and tail written here; the final avalanche is
    the oracle's fmix32, so the published vectors pin it."""
    c1, c2 = 0xCC9E2D51, 0x1B873593

    def rot(x, r):
        return ((x << r) | (x >> (32 - r))) & M32

    h = seed & M32
    n = len(key)
    nb = n - n % 4
    for i in range(0, nb, 4):
        k = int.from_bytes(key[i:i + 4], "little")
        k = (k * c1) & M32
        k = rot(k, 15)
        k = (k * c2) & M32
        h ^= k
        h = rot(h, 13)
        h = (h * 5 + 0xE6546B64) & M32
    tail = key[nb:]
    if tail:
        k = 0
        for j, b in enumerate(tail):
            k |= b << (8 * j)
        k = (k * c1) & M32
        k = rot(k, 15)
        k = (k * c2) & M32
        h ^= k
    h ^= n
    return oracle.fmix32(h)


def read_murmur_vectors():
    out = []
    with open(os.path.join(GOLDEN, "murmur3_x86_32_vectors.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key_hex, seed_hex, h_hex = line.split()
            key = b"" if key_hex == "-" else bytes.fromhex(key_hex)
            out.append((key, int(seed_hex, 16), int(h_hex, 16)))
    return out


def rotl_closed(x: int, k: int) -> int:
    k %= 32
    if k == 0:
        return x
    return (x * 2 ** k) % 2 ** 32 + x // 2 ** (32 - k)


def single_run(oracle, *, words, outcomes, table, thr, n_routes, route_mode=ROUTE_MOD,
               cdf=None, n_steps=1, step0=0, sizes=None, ld=None, decisions=None, record=False):
    """Run the oracle over sessions whose initial words/outcomes are given.

    ``words``: [N][W] python ints; ``outcomes``: [N]."""
    N = len(words)
    W = len(words[0])
    ld = N if ld is None else ld
    state = np.zeros((W, ld), dtype=np.uint32)
    state[:, :N] = np.asarray(words, dtype=np.uint64).T.astype(np.uint32)
    outcome = np.zeros(ld, dtype=np.uint32)
    outcome[:N] = np.asarray(outcomes, dtype=np.uint64).astype(np.uint32)
    sizes = [N] if sizes is None else sizes
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    return oracle.run_chain(n_words=W, n_routes=n_routes, cohort_offsets=offsets,
                            table=np.asarray(table, dtype=np.uint32).reshape(n_routes, 16),
                            route_mode=route_mode, route_cdf=cdf, decide_thr=thr,
                            state=state, outcome=outcome, n_steps=n_steps, step0=step0,
                            decisions=decisions, record=record)


def rand_u32(n, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)


# --------------------------------------------------------------------------
# pins: primitives
# --------------------------------------------------------------------------
def pin_fmix32_vectors(oracle):
    for key, seed, want in read_murmur_vectors():
        got = murmur3_x86_32(oracle, key, seed)
        assert got == want, "murmur3(%r, %#x) = %#x, published %#x" % (key, seed, got, want)


def pin_rotl_closed_form(oracle):
    for x in SPECIAL + [int(v) for v in rand_u32(16, 1)]:
        for k in range(0, 70):
            assert oracle.rotl(x, k) == rotl_closed(x, k), (x, k)
    # applying rotl by k, 32/gcd(k,32) times, is the identity
    for k in range(1, 32):
        x = 0x9E3779B9
        for _ in range(32 // math.gcd(k, 32)):
            x = oracle.rotl(x, k)
        assert x == 0x9E3779B9, k


def pin_route_mod(oracle):
    for R in (1, 3, 4, 5, 16, 17, 256, 1000, 1024):
        counts = oracle.route_histogram(0, 1 << 20, R, ROUTE_MOD)
        want = np.asarray([len(range(r, 1 << 20, R)) for r in range(R)], dtype=np.uint64)
        assert np.array_equal(counts, want), R
        for o in SPECIAL:
            assert oracle.route(o, R, ROUTE_MOD) == o % R, (o, R)


def _cdf_cases():
    z = lambda R, s: (lambda w: np.minimum(np.floor(np.cumsum(w)[:-1] / np.sum(w) * 2.0 ** 32), M32).astype(np.uint32))(
        np.arange(1, R + 1, dtype=np.float64) ** (-s))
    return [
        np.asarray([0x40000000, 0x80000000, 0xC0000000], dtype=np.uint32),
        np.asarray([0, 0, 5, 5, 5, 0xFFFFFFFF], dtype=np.uint32),  # ties and extremes
        np.asarray([1, 0x100], dtype=np.uint32),
        z(64, 1.1), z(1024, 1.1),
    ]


def pin_route_cdf(oracle):
    for cdf in _cdf_cases():
        R = cdf.size + 1
        # closed form: route = number of thresholds not above o
        probes = set(SPECIAL)
        for v in cdf.tolist():
            for d in (-1, 0, 1):
                if 0 <= v + d <= M32:
                    probes.add(v + d)
        for o in sorted(probes):
            want = int(np.sum(cdf.astype(np.uint64) <= o))
            assert oracle.route(o, R, ROUTE_CDF, cdf) == want, (o, R)
        # exact histogram over a window: counts are interval intersections
        if R <= 64:
            lo, hi = 0, 1 << 18
            counts = oracle.route_histogram(lo, hi, R, ROUTE_CDF, cdf)
            edges = [0] + [int(v) for v in cdf] + [1 << 32]
            want = [max(0, min(hi, edges[k + 1]) - max(lo, edges[k])) for k in range(R)]
            assert counts.tolist() == want, R


def pin_decide_known_answers(oracle):
    # fmix32(0) = 0, fmix32(1) = 0x514E28B7 (low half 0x28B7),
    # fmix32(0xFFFFFFFF) = 0x81F16F39 (low half 0x6F39): published values.
    for key, low in ((0, 0), (1, 0x28B7), (0xFFFFFFFF, 0x6F39)):
        for s0, o, step in ((key, 0, 0), (0, key, 0), (0, 0, key),
                            (key ^ 0x5555AAAA, 0x5555AAAA, 0), (0x0F0F0F0F, key ^ 0x0F0F0F0F ^ 77, 77)):
            assert oracle.decide(s0, o, step, low) == 0, (s0, o, step)
            assert oracle.decide(s0, o, step, low + 1) == 1, (s0, o, step)
            assert oracle.decide(s0, o, step, 0) == 0
            assert oracle.decide(s0, o, step, 65536) == 1


def pin_decision_rate_exhaustive(oracle, cases=((0x12345678, 3, 19661), (0, 0, 3277))):
    """Over all 2^32 outcomes exactly thr * 65536 are taken (bijection)."""
    from concurrent.futures import ThreadPoolExecutor  # ctypes drops the GIL

    with ThreadPoolExecutor(max_workers=len(cases)) as ex:
        counts = list(ex.map(lambda c: oracle.count_taken_all_outcomes(*c), cases))
    for (s0, step, thr), n in zip(cases, counts):
        assert n == thr * 65536, (s0, step, thr, n)


# --------------------------------------------------------------------------
# pins: route bodies in closed form
# --------------------------------------------------------------------------
def pin_taken_unit_table(oracle):
    """thr = 65536 (always taken), table of ones, zero state: S'[w] = w + 1."""
    W = 64
    res = single_run(oracle, words=[[0] * W], outcomes=[12345], table=[1] * 16, thr=65536,
                     n_routes=1)
    assert res["state"][:, 0].tolist() == [w + 1 for w in range(W)]
    assert res["eff_payload"][0, 0, :].tolist() == [1, 2, 3, 4]
    assert res["n_taken"][0, 0] == 1


def pin_taken_single_column(oracle):
    """Only table column j nonzero: S'[w] = (w + 1) * v where w = j mod 16."""
    W = 64
    for j, v in ((0, 1), (5, 3), (15, 0x80000001)):
        row = [0] * 16
        row[j] = v
        x0 = 0x0F0F0F0F
        res = single_run(oracle, words=[[x0] * W], outcomes=[7], table=row, thr=65536, n_routes=1)
        want = [x0 ^ (((w + 1) * v) % 2 ** 32) if w % 16 == j else x0 for w in range(W)]
        assert res["state"][:, 0].tolist() == want, j


def pin_taken_involution(oracle):
    """R = 1, always taken: two steps XOR the same mask, so even T restores
    the state, whatever the outcomes."""
    rng_words = rand_u32(6 * 20, 11).reshape(6, 20)
    table = rand_u32(16, 12)
    res = single_run(oracle, words=rng_words.tolist(), outcomes=rand_u32(6, 13).tolist(),
                     table=table, thr=65536, n_routes=1, n_steps=4, sizes=[2, 4])
    assert np.array_equal(res["state"][:, :6], rng_words.T), "even T must restore"
    assert res["n_taken"].tolist() == [[2, 4]] * 4


def pin_not_taken_rotation(oracle):
    """thr = 0 (never taken), R = 1, outcome forced to 0 before each step:
    S_{t+1} = rotl(S_t, 1); 32 steps restore the state."""
    words = [[1, 0x80000000, 0xDEADBEEF, 0xFFFFFFFF, 0x12345678]]
    state = np.asarray(words, dtype=np.uint32).T.copy()
    outcome = np.zeros(1, dtype=np.uint32)
    offsets = np.asarray([0, 1], dtype=np.uint32)
    table = rand_u32(16, 3).reshape(1, 16)
    first = None
    for t in range(32):
        outcome[:] = 0
        oracle.run_chain(n_words=5, n_routes=1, cohort_offsets=offsets, table=table,
                         route_mode=ROUTE_MOD, route_cdf=None, decide_thr=0, state=state,
                         outcome=outcome, n_steps=1, step0=t)
        if first is None:
            first = state[:, 0].tolist()
    assert first == [rotl_closed(x, 1) for x in words[0]]
    assert state[:, 0].tolist() == words[0]


def pin_not_taken_amounts(oracle):
    """Never taken, MOD routes: S' = rotl(S, (r + 1) mod 32) + o, o = r."""
    R = 40
    for r in range(R):
        o = r
        words = [[1, 0x80000000, 0xFFFFFFFF, 0x00010000]]
        res = single_run(oracle, words=words, outcomes=[o], table=rand_u32(R * 16, 5), thr=0,
                         n_routes=R)
        want = [(rotl_closed(x, (r + 1) % 32) + o) % 2 ** 32 for x in words[0]]
        assert res["state"][:, 0].tolist() == want, r
    # (r + 1) = 32: rotation is the identity, the body only adds the outcome
    res = single_run(oracle, words=[[5, 0xFFFFFFFF, 7, 9]], outcomes=[31 + 32 * 1000],
                     table=rand_u32(32 * 16, 6), thr=0, n_routes=32)
    o = 31 + 32 * 1000
    assert res["state"][:, 0].tolist() == [(x + o) % 2 ** 32 for x in (5, 0xFFFFFFFF, 7, 9)]


def pin_cdf_route_in_chain(oracle):
    """CDF route keys reach the body: never taken, S = 1 gives 2^(r+1) + o."""
    cdf = np.asarray([100, 200, 200, 1000], dtype=np.uint32)
    for o, r in ((0, 0), (99, 0), (100, 1), (199, 1), (200, 3), (999, 3), (1000, 4), (M32, 4)):
        res = single_run(oracle, words=[[1, 1, 1, 1]], outcomes=[o], table=rand_u32(5 * 16, 8),
                         thr=0, n_routes=5, route_mode=ROUTE_CDF, cdf=cdf)
        assert res["state"][0, 0] == (2 ** (r + 1) + o) % 2 ** 32, (o, r)


def pin_tool_column(oracle):
    """tool = table[r][d] mod 8: column 1 when taken, column 0 when not."""
    R = 4
    table = np.zeros((R, 16), dtype=np.uint32)
    for r in range(R):
        table[r, 0] = 8 * 1000 + r          # tool r when not taken
        table[r, 1] = 8 * 77 + (7 - r)      # tool 7-r when taken
    for r in range(R):
        for thr, want in ((0, r), (65536, 7 - r)):
            res = single_run(oracle, words=[[3, 4, 5, 6]], outcomes=[r + 4 * 9], table=table,
                             thr=thr, n_routes=R)
            assert res["eff_tool"][0, 0] == want, (r, thr)


# --------------------------------------------------------------------------
# pins: decision inputs, payload, compaction, chaining
# --------------------------------------------------------------------------
def pin_decide_uses_pre_update_state_and_step(oracle):
    """fmix32(0) = 0 (published), so with S[0] ^ o ^ step = 0 the decision is
    taken for thr = 1 and for no smaller threshold.  Build a two-step chain
    in which this holds at both steps only if the decision reads the
    pre-update word, step = step0 + t, and the next outcome fmix32(S'[0])."""
    table = [0] * 16  # the taken body then leaves the state unchanged
    for s0 in (0x0BADF00D, 0xFFFFFFFF, 1):
        o1 = murmur3_x86_32(oracle, b"", s0)          # = fmix32(s0)
        step0 = ((s0 ^ o1) - 1) % 2 ** 32              # step 1 then gives 0
        o0 = s0 ^ step0                                # step 0 gives 0
        res = single_run(oracle, words=[[s0, 5, 6, 7]], outcomes=[o0], table=table, thr=1,
                         n_routes=1, n_steps=2, step0=step0)
        assert res["n_taken"][:, 0].tolist() == [1, 1], s0
        res = single_run(oracle, words=[[s0, 5, 6, 7]], outcomes=[o0 ^ 1], table=table, thr=1,
                         n_routes=1, n_steps=1, step0=step0)
        assert res["n_taken"][0, 0] == 0  # fmix32(1) has low half 0x28B7 >= 1
    # a taken step with a nonzero mask changes S[0]; the decision must still
    # come from the word before the update (S0 ^ o ^ step = 0 -> taken)
    res = single_run(oracle, words=[[0x55, 1, 2, 3]], outcomes=[0x55 ^ 9], table=[0xFFFF] * 16,
                     thr=1, n_routes=1, step0=9)
    assert res["n_taken"][0, 0] == 1


def pin_payload_post_update(oracle):
    """The emitted payload is the state after the update (taken, unit table:
    1, 2, 3, 4 from a zero state; not taken: rotl(0) + o = o)."""
    res = single_run(oracle, words=[[0] * 8], outcomes=[9], table=[1] * 16, thr=65536, n_routes=1)
    assert res["eff_payload"][0, 0, :].tolist() == [1, 2, 3, 4]
    res = single_run(oracle, words=[[0] * 8], outcomes=[9], table=[1] * 16, thr=0, n_routes=1)
    assert res["eff_payload"][0, 0, :].tolist() == [9, 9, 9, 9]


def _decisions_by_pinned_rule(oracle, s0, o, step, thr):
    return oracle.decide(int(s0), int(o), step, thr)


def pin_stable_partition(oracle):
    """Effects of each cohort are ordered by Python's stable sort with key
    (not taken, sid); taken-ness from the (pinned) decide rule."""
    sizes = [1, 2, 7, 33, 64, 65, 100, 256, 3]
    N = sum(sizes)
    words = rand_u32(N * 4, 21).reshape(N, 4)
    outs = rand_u32(N, 22)
    for thr in (1, 19661, 32768, 65535):
        res = single_run(oracle, words=words.tolist(), outcomes=outs.tolist(),
                         table=rand_u32(16 * 8, 23), thr=thr, n_routes=8, sizes=sizes, step0=5)
        offs = np.concatenate([[0], np.cumsum(sizes)])
        for c in range(len(sizes)):
            members = list(range(offs[c], offs[c + 1]))
            d = {s: oracle.decide(int(words[s, 0]), int(outs[s]), 5, thr) for s in members}
            want = sorted(members, key=lambda s: (not d[s], s))
            got = res["eff_sid"][0, offs[c]:offs[c + 1]].tolist()
            assert got == want, (thr, c)
            assert res["n_taken"][0, c] == sum(d.values())


def pin_chain_invariants(oracle):
    """Counts, coverage and chaining over a multi-cohort, multi-step run."""
    sizes = [5, 64, 1, 256, 17, 128]
    N, W, T, R = sum(sizes), 12, 6, 7
    words = rand_u32(N * W, 31).reshape(N, W)
    outs = rand_u32(N, 32)
    ld = N + 9
    res = single_run(oracle, words=words.tolist(), outcomes=outs.tolist(),
                     table=rand_u32(R * 16, 33), thr=32768, n_routes=R, sizes=sizes,
                     n_steps=T, step0=1000, ld=ld)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    sid = res["eff_sid"]
    pay = res["eff_payload"]
    for t in range(T):
        for c in range(len(sizes)):
            seg = sid[t, offs[c]:offs[c + 1]]
            assert sorted(seg.tolist()) == list(range(offs[c], offs[c + 1]))  # each sid once
            assert 0 <= res["n_taken"][t, c] <= sizes[c]
        # padding slots never written
        assert np.all(sid[t, N:] == 0xFFFFFFFF) and np.all(pay[t, N:, :] == 0xFFFFFFFF)
    # total effects = N * T
    assert int(np.sum(sid[:, :N] != 0xFFFFFFFF)) == N * T
    # O_{t+1} = fmix32(payload_t[0]) and the last payload is the final state
    pos = {}
    for t in range(T):
        pos[t] = np.empty(N, dtype=np.int64)
        pos[t][sid[t, :N]] = np.arange(N)
    for s in range(0, N, 7):
        assert pay[T - 1, pos[T - 1][s], :].tolist() == res["state"][:4, s].tolist()
        assert res["outcome"][s] == pyref.fmix32(int(pay[T - 1, pos[T - 1][s], 0]))
    # padding columns of state / outcome untouched
    assert np.all(res["state"][:, N:] == 0) and np.all(res["outcome"][N:] == 0)


def pin_untouched_outside_range(oracle):
    sizes = [10, 20, 30, 40]
    N, W, R = sum(sizes), 6, 3
    words = rand_u32(N * W, 41).reshape(W, N)
    outs = rand_u32(N, 42)
    state = words.copy()
    outcome = outs.copy()
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    res = oracle.run_chain(n_words=W, n_routes=R, cohort_offsets=offsets,
                           table=rand_u32(R * 16, 43), route_mode=ROUTE_MOD, route_cdf=None,
                           decide_thr=32768, state=state, outcome=outcome, n_steps=3,
                           cohort_begin=1, cohort_end=3)
    a, b = offsets[1], offsets[3]
    assert np.array_equal(state[:, :a], words[:, :a]) and np.array_equal(state[:, b:], words[:, b:])
    assert np.array_equal(outcome[:a], outs[:a]) and np.array_equal(outcome[b:], outs[b:])
    assert not np.array_equal(state[:, a:b], words[:, a:b])
    assert np.all(res["eff_sid"][:, :a] == 0xFFFFFFFF) and np.all(res["eff_sid"][:, b:] == 0xFFFFFFFF)
    assert np.all(res["n_taken"][:, [0, 3]] == 0xFFFFFFFF)


def pin_chain_composes(oracle):
    """run(T1, step0) then run(T2, step0 + T1) equals run(T1 + T2, step0)."""
    sizes = [32, 64, 3]
    N, W, R = sum(sizes), 9, 5
    words = rand_u32(N * W, 51).reshape(W, N)
    outs = rand_u32(N, 52)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    table = rand_u32(R * 16, 53)
    kw = dict(n_words=W, n_routes=R, cohort_offsets=offsets, table=table, route_mode=ROUTE_CDF,
              route_cdf=np.asarray([1 << 30, 1 << 31, 3 << 30, 0xF0000000], dtype=np.uint32),
              decide_thr=19661)
    s1, o1 = words.copy(), outs.copy()
    full = oracle.run_chain(state=s1, outcome=o1, n_steps=7, step0=10, **kw)
    s2, o2 = words.copy(), outs.copy()
    a = oracle.run_chain(state=s2, outcome=o2, n_steps=3, step0=10, **kw)
    b = oracle.run_chain(state=s2, outcome=o2, n_steps=4, step0=13, **kw)
    assert np.array_equal(s1, s2) and np.array_equal(o1, o2)
    assert np.array_equal(full["eff_sid"], np.concatenate([a["eff_sid"], b["eff_sid"]]))
    assert np.array_equal(full["eff_payload"], np.concatenate([a["eff_payload"], b["eff_payload"]]))
    assert np.array_equal(full["n_taken"], np.concatenate([a["n_taken"], b["n_taken"]]))


def pin_replay_deterministic(oracle):
    sizes = [64, 64, 7]
    N, W, R = sum(sizes), 16, 16
    words = rand_u32(N * W, 61).reshape(W, N)
    outs = rand_u32(N, 62)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    runs = []
    for _ in range(2):
        st, oc = words.copy(), outs.copy()
        r = oracle.run_chain(n_words=W, n_routes=R, cohort_offsets=offsets,
                             table=rand_u32(R * 16, 63), route_mode=ROUTE_MOD, route_cdf=None,
                             decide_thr=32768, state=st, outcome=oc, n_steps=8)
        runs.append((st.tobytes(), oc.tobytes(), r["eff_sid"].tobytes(),
                     r["eff_payload"].tobytes(), r["n_taken"].tobytes()))
    assert runs[0] == runs[1]


# --------------------------------------------------------------------------
# brute force against the independent Python formulation
# --------------------------------------------------------------------------
def pin_brute_force_tiny(oracle, quick=False):
    """Every (state, outcome) pair of a tiny domain, every route and both
    decisions, compared session by session with the Python formulation."""
    vals = [0, 1, 0x80000000, 0xFFFFFFFF] if quick else [0, 1, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF]
    W = 4
    for R, mode in ((4, ROUTE_MOD), (5, ROUTE_CDF), (33, ROUTE_MOD)):
        cdf = np.asarray([0x10, 0x80000000, 0x80000001, 0xFFFFFFF0], dtype=np.uint32) \
            if mode == ROUTE_CDF else None
        table = rand_u32(R * 16, 70 + R).reshape(R, 16)
        states = list(itertools.product(vals, repeat=W))
        outs = [0, 1, 2, 3, 4, 31, 32, 0x10, 0x80000000, 0x80000001, 0xFFFFFFF0, 0xFFFFFFFF]
        pairs = [(s, o) for s in states for o in outs]
        for thr in ((32768,) if quick else (0, 1, 32768, 65535, 65536)):
            for step0 in ((0,) if quick else (0, 1, 0xFFFFFFFF)):
                words = [list(s) for s, _ in pairs]
                res = single_run(oracle, words=words, outcomes=[o for _, o in pairs], table=table,
                                 thr=thr, n_routes=R, route_mode=mode, cdf=cdf, step0=step0,
                                 sizes=[1] * len(pairs), n_steps=2)
                sess = {i: list(s) for i, (s, _) in enumerate(pairs)}
                outd = {i: o for i, (_, o) in enumerate(pairs)}
                p_s, p_o, p_e, p_c = pyref.run_chain(
                    sess, outd, [[i] for i in range(len(pairs))], 2, step0, R, table.tolist(),
                    mode, [] if cdf is None else cdf.tolist(), thr)
                got_state = res["state"].T.tolist()
                for i in range(len(pairs)):
                    assert got_state[i] == p_s[i], (R, thr, step0, pairs[i])
                    assert res["outcome"][i] == p_o[i]
                    for t in range(2):
                        (sid, tool, pay), = p_e[t][i]
                        assert res["eff_sid"][t, i] == sid and res["eff_tool"][t, i] == tool
                        assert tuple(res["eff_payload"][t, i, :].tolist()) == pay
                        assert res["n_taken"][t, i] == p_c[t][i]


def pin_brute_force_cohorts(oracle):
    """Multi-session cohorts (compaction) against the Python formulation."""
    sizes = [1, 2, 3, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256]
    N, W, R = sum(sizes), 5, 6
    words = rand_u32(N * W, 81).reshape(N, W)
    outs = rand_u32(N, 82)
    table = rand_u32(R * 16, 83).reshape(R, 16)
    cdf = np.asarray([100, 1 << 28, 1 << 30, 1 << 31, 0xF0000000], dtype=np.uint32)
    for mode in (ROUTE_MOD, ROUTE_CDF):
        res = single_run(oracle, words=words.tolist(), outcomes=outs.tolist(), table=table,
                         thr=19661, n_routes=R, route_mode=mode,
                         cdf=cdf if mode == ROUTE_CDF else None, sizes=sizes, n_steps=3, step0=2)
        offs = np.concatenate([[0], np.cumsum(sizes)])
        cohorts = [list(range(offs[c], offs[c + 1])) for c in range(len(sizes))]
        p_s, p_o, p_e, p_c = pyref.run_chain(
            {i: words[i].tolist() for i in range(N)}, {i: int(outs[i]) for i in range(N)},
            cohorts, 3, 2, R, table.tolist(), mode, cdf.tolist() if mode == ROUTE_CDF else [],
            19661)
        assert res["state"].T.tolist() == [p_s[i] for i in range(N)]
        assert res["outcome"].tolist() == [p_o[i] for i in range(N)]
        for t in range(3):
            for c, members in enumerate(cohorts):
                e = p_e[t][c]
                sl = slice(offs[c], offs[c + 1])
                assert res["eff_sid"][t, sl].tolist() == [x[0] for x in e]
                assert res["eff_tool"][t, sl].tolist() == [x[1] for x in e]
                assert res["eff_payload"][t, sl, :].tolist() == [list(x[2]) for x in e]
                assert res["n_taken"][t, c] == p_c[t][c]


# --------------------------------------------------------------------------
# pins: the no-decision floor (Section 7 "Matched mechanisms": the recorded
# route sequence replayed without predicate or selection)
# --------------------------------------------------------------------------
def bits_from_bool(dec):
    """[T][ld] booleans -> [T][ceil(ld/32)] uint32 bitmap, bit s mod 32 of
    word s // 32 (written with plain Python integers)."""
    T, ld = len(dec), len(dec[0])
    out = np.zeros((T, (ld + 31) // 32), dtype=np.uint32)
    for t in range(T):
        for s in range(ld):
            if dec[t][s]:
                out[t, s // 32] = int(out[t, s // 32]) | (1 << (s % 32))
    return out


def pin_floor_replays_recorded(oracle):
    """The chain's recorded decisions replayed through the floor give the
    chain's outputs; the record agrees with the pinned decision rule and with
    the taken counts."""
    sizes = [5, 32, 33, 64, 70]
    N, W, R, ld = sum(sizes), 6, 7, sum(sizes) + 9
    words = rand_u32(N * W, 301).reshape(N, W).tolist()
    outs = rand_u32(N, 302).tolist()
    table = rand_u32(R * 16, 303).reshape(R, 16)
    base = single_run(oracle, words=words, outcomes=outs, table=table, thr=30000, n_routes=R,
                      sizes=sizes, ld=ld, n_steps=4, step0=11)
    rec = single_run(oracle, words=words, outcomes=outs, table=table, thr=30000, n_routes=R,
                     sizes=sizes, ld=ld, n_steps=1, step0=11, record=True)["decisions"]
    for s in range(N):
        want = _decisions_by_pinned_rule(oracle, words[s][0], outs[s], 11, 30000)
        assert ((int(rec[0, s // 32]) >> (s % 32)) & 1) == want
    for s in range(N, ld):  # sessions past N are never stepped
        assert ((int(rec[0, s // 32]) >> (s % 32)) & 1) == 0
    full = single_run(oracle, words=words, outcomes=outs, table=table, thr=30000, n_routes=R,
                      sizes=sizes, ld=ld, n_steps=4, step0=11, record=True)
    flo = single_run(oracle, words=words, outcomes=outs, table=table, thr=0, n_routes=R,
                     sizes=sizes, ld=ld, n_steps=4, step0=999, decisions=full["decisions"])
    for k in base:
        assert np.array_equal(base[k], flo[k]), k
    offs = np.concatenate([[0], np.cumsum(sizes)])
    for t in range(4):
        for c in range(len(sizes)):
            n = sum((int(full["decisions"][t, s // 32]) >> (s % 32)) & 1 for s in range(offs[c], offs[c + 1]))
            assert n == int(base["n_taken"][t, c])


def pin_floor_against_pyref(oracle):
    """Random decision bitmaps (every cohort size class, both route maps)
    against the Python formulation with the same forced decisions."""
    sizes = [1, 3, 31, 32, 33, 64, 65, 129, 256]
    N, W, R, T = sum(sizes), 5, 6, 3
    ld = N + 5
    words = rand_u32(N * W, 311).reshape(N, W)
    outs = rand_u32(N, 312)
    table = rand_u32(R * 16, 313).reshape(R, 16)
    cdf = np.asarray([7, 1 << 27, 1 << 30, 3 << 30, 0xFFFFFFF0], dtype=np.uint32)
    rng = np.random.Generator(np.random.PCG64(314))
    dec = (rng.random((T, ld)) < 0.37).tolist()
    bits = bits_from_bool(dec)
    offs = np.concatenate([[0], np.cumsum(sizes)])
    cohorts = [list(range(offs[c], offs[c + 1])) for c in range(len(sizes))]
    for mode in (ROUTE_MOD, ROUTE_CDF):
        res = single_run(oracle, words=words.tolist(), outcomes=outs.tolist(), table=table,
                         thr=12345, n_routes=R, route_mode=mode, cdf=cdf if mode == ROUTE_CDF else None,
                         sizes=sizes, n_steps=T, ld=ld, decisions=bits)
        p_s, p_o, p_e, p_c = pyref.run_chain(
            {i: words[i].tolist() for i in range(N)}, {i: int(outs[i]) for i in range(N)},
            cohorts, T, 0, R, table.tolist(), mode, cdf.tolist() if mode == ROUTE_CDF else [],
            12345, forced=lambda t, s: dec[t][s])
        assert res["state"][:, :N].T.tolist() == [p_s[i] for i in range(N)]
        assert res["outcome"][:N].tolist() == [p_o[i] for i in range(N)]
        for t in range(T):
            for c in range(len(sizes)):
                e = p_e[t][c]
                sl = slice(offs[c], offs[c + 1])
                assert res["eff_sid"][t, sl].tolist() == [x[0] for x in e]
                assert res["eff_tool"][t, sl].tolist() == [x[1] for x in e]
                assert res["eff_payload"][t, sl, :].tolist() == [list(x[2]) for x in e]
                assert res["n_taken"][t, c] == p_c[t][c]


def pin_floor_closed_forms(oracle):
    """All taken on one route: two steps XOR the same masks, so the state
    returns after every even number of steps whatever the threshold, and
    every session is counted; none taken with outcome 0 for one step: every
    word is rotated left by 1."""
    N, W, ld = 70, 8, 96
    words = rand_u32(N * W, 321).reshape(N, W).tolist()
    outs = rand_u32(N, 322).tolist()
    table = rand_u32(16, 323).reshape(1, 16)
    ones = np.full((4, ld // 32), 0xFFFFFFFF, dtype=np.uint32)
    res = single_run(oracle, words=words, outcomes=outs, table=table, thr=0, n_routes=1,
                     n_steps=4, ld=ld, decisions=ones)
    assert res["state"][:, :N].T.tolist() == words
    assert res["n_taken"][:, 0].tolist() == [N] * 4
    assert res["eff_sid"][:, :N].tolist() == [list(range(N))] * 4
    zeros = np.zeros((1, ld // 32), dtype=np.uint32)
    res = single_run(oracle, words=words, outcomes=[0] * N, table=table, thr=65536, n_routes=1,
                     n_steps=1, ld=ld, decisions=zeros)
    assert res["state"][:, :N].T.tolist() == [[rotl_closed(x, 1) for x in w] for w in words]
    assert res["n_taken"][0, 0] == 0


QUICK_PINS = [
    pin_fmix32_vectors, pin_rotl_closed_form, pin_route_mod, pin_route_cdf,
    pin_decide_known_answers, pin_taken_unit_table, pin_taken_single_column,
    pin_taken_involution, pin_not_taken_rotation, pin_not_taken_amounts,
    pin_cdf_route_in_chain, pin_tool_column, pin_decide_uses_pre_update_state_and_step,
    pin_payload_post_update, pin_stable_partition, pin_chain_invariants,
    pin_untouched_outside_range, pin_chain_composes, pin_replay_deterministic,
    pin_floor_replays_recorded, pin_floor_against_pyref, pin_floor_closed_forms,
]
