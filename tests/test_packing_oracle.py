"""The packing oracle (F, P*, U) pinned on the CPU.

Pins: exhaustive search over every feasible schedule on tiny instances, the
inclusive deadline boundary, witness validity, the ordering F <= P* <= U
(Section 3, Proposition "Boundary ordering"), the five validity gates of
Section 5 ("Prospective freeze and validity gates": ordering, monotone under
grouping coarsening, monotone in delta, antitone in K, equality when the
bounds coincide), closed forms, and U recomputed over every integer launch
time of a tiny clock.  Planted mistakes in a copy of the oracle are caught.
"""
import importlib.util
import random

import pytest

from oracle import packing as PK


def rand_instance(rng, n, n_routes, span):
    t = [rng.randrange(span) for _ in range(n)]
    r = [rng.randrange(n_routes) for _ in range(n)]
    return t, r


def test_exact_packing_equals_exhaustive_search():
    rng = random.Random(2026)
    for trial in range(400):
        n = rng.randrange(1, 9)
        R = rng.randrange(1, 4)
        t, r = rand_instance(rng, n, R, rng.choice([4, 10, 30]))
        K = [rng.randrange(1, 4) for _ in range(R)] if trial % 2 else rng.randrange(1, 4)
        delta = rng.randrange(0, 12)
        p, w = PK.exact_packing(t, r, K, delta)
        assert p == PK.brute_force_packing(t, r, K, delta), (t, r, K, delta)


def test_inclusive_deadline_boundary():
    # two events exactly delta apart share a launch time; delta + 1 apart do not
    assert PK.exact_packing([0, 50], [0, 0], 2, 50)[0] == 2
    assert PK.exact_packing([0, 51], [0, 0], 2, 50)[0] == 0
    assert PK.local_overlap([0, 50], [0, 0], 2, 50) == 2
    assert PK.local_overlap([0, 51], [0, 0], 2, 50) == 0
    # fixed windows are half-open: 49 and 50 fall in different windows of 50
    assert PK.fixed_eligible([0, 49], [0, 0], 2, 50) == 2
    assert PK.fixed_eligible([49, 50], [0, 0], 2, 50) == 0
    # a chain a-b-c with gaps of delta: only one pair can launch together
    assert PK.exact_packing([0, 10, 20], [0, 0, 0], 2, 10)[0] == 2
    assert PK.exact_packing([0, 10, 20, 30], [0, 0, 0, 0], 2, 10)[0] == 4


def test_witness_is_a_feasible_disjoint_schedule_of_size_p_star():
    rng = random.Random(7)
    for _ in range(60):
        R = rng.randrange(1, 5)
        t, r = rand_instance(rng, rng.randrange(20, 120), R, 1000)
        K = [rng.randrange(1, 6) for _ in range(R)]
        delta = rng.randrange(5, 200)
        p, w = PK.exact_packing(t, r, K, delta)
        seen = set()
        for b in w:
            assert PK.batch_is_feasible(b, t, r, K, delta)
            assert not (seen & set(b))
            seen |= set(b)
        assert len(seen) == p


def test_ordering_and_equality_gate():
    rng = random.Random(11)
    for _ in range(60):
        R = rng.randrange(1, 5)
        t, r = rand_instance(rng, rng.randrange(10, 150), R, rng.choice([300, 3000]))
        K = rng.randrange(1, 8)
        delta = rng.randrange(1, 400)
        f, p, u, _ = PK.shares(t, r, K, delta, origin=rng.randrange(0, delta))
        assert f <= p <= u, (f, p, u)
        if f == u:
            assert p == f


def test_monotone_gates():
    rng = random.Random(13)
    for _ in range(40):
        t, r = rand_instance(rng, rng.randrange(20, 100), 4, 2000)
        delta = rng.randrange(10, 300)
        base = PK.shares(t, r, 3, delta)[:3]
        # grouping coarsening: routes {0,1} and {2,3} merged
        coarse = [x // 2 for x in r]
        c = PK.shares(t, coarse, 3, delta)[:3]
        assert all(a <= b for a, b in zip(base, c)), (base, c)
        # larger delta: P* and U cannot shrink; F cannot shrink when the
        # windows nest (2 delta, same origin)
        d2 = PK.shares(t, r, 3, 2 * delta)[:3]
        assert all(a <= b for a, b in zip(base, d2)), (base, d2)
        # larger K: no share can grow
        k4 = PK.shares(t, r, 4, delta)[:3]
        assert all(a >= b for a, b in zip(base, k4)), (base, k4)


def test_closed_forms():
    # n simultaneous events on one route: everything or nothing
    for n in (1, 5, 9):
        for K in (1, 5, 6):
            want = n if n >= K else 0
            assert PK.exact_packing([7] * n, [3] * n, K, 0)[0] == want
            assert PK.local_overlap([7] * n, [3] * n, K, 0) == want
            assert PK.fixed_eligible([7] * n, [3] * n, K, 10) == want
    # evenly spaced releases, spacing s, delta = m s: every release opens a
    # window of m + 1 events, so with K <= m + 1 every event is packed
    t = [5 * i for i in range(40)]
    assert PK.exact_packing(t, [0] * 40, 4, 15)[0] == 40
    assert PK.exact_packing(t, [0] * 40, 5, 15)[0] == 0


def test_local_overlap_against_every_integer_launch_time():
    rng = random.Random(17)
    for _ in range(100):
        R = rng.randrange(1, 3)
        t, r = rand_instance(rng, rng.randrange(1, 12), R, 40)
        K = rng.randrange(1, 5)
        delta = rng.randrange(0, 15)
        want = 0
        for ti, ri in zip(t, r):
            best = max(sum(1 for tj, rj in zip(t, r) if rj == ri and tj <= tau <= tj + delta)
                       for tau in range(ti, ti + delta + 1))
            want += best >= K
        assert PK.local_overlap(t, r, K, delta) == want


MUTANTS = {
    "strict_deadline": ("if ts[j - 1] - ts[i - 1] <= delta:", "if ts[j - 1] - ts[i - 1] < delta:"),
    "k_off_by_one": ("for i in range(1, j - k + 2):", "for i in range(1, j - k + 1):"),
    "dp_wrong_prefix": ("cand = D[i - 1] + j - i + 1", "cand = D[i] + j - i"),
    "dp_no_carry": ("            D[j] = D[j - 1]\n", "            D[j] = 0\n"),
    "fixed_closed_windows": ("w = (int(ti) - origin) // delta", "w = (int(ti) - origin + delta - 1) // delta"),
    "fixed_ge_strict": ("if n >= _k(K, rr))", "if n > _k(K, rr))"),
    "overlap_open_end": ("if tj <= tau <= tj + delta)", "if tj <= tau < tj + delta)"),
    "overlap_only_own_time": ("cands = [ti] + [tj for tj in same if ti <= tj <= ti + delta]", "cands = [ti]"),
}


def _pins(mod):
    global PK
    saved = PK
    PK = mod
    try:
        test_exact_packing_equals_exhaustive_search()
        test_inclusive_deadline_boundary()
        test_closed_forms()
        test_local_overlap_against_every_integer_launch_time()
        test_ordering_and_equality_gate()
    finally:
        PK = saved


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_packing_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(PK.__file__).read()
    assert src.count(old) == 1, "anchor not found: %s" % name
    path = tmp_path / ("packing_%s.py" % name)
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location("packing_" + name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    with pytest.raises(AssertionError):
        _pins(mod)
