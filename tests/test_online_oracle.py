"""The online-compactor oracle pinned on the CPU.

Pins: a second formulation of the same frozen policy that walks every integer
time of a tiny clock (arrivals of the tick first, then the triggers due at
that tick); A <= P* against the packing oracle (Eq. ordering, which the
exhaustive-search-pinned packing oracle stands behind); every launched batch
feasible (Eq. feasible-batch with the launch latency) and within capacity;
the event count conserved; closed forms; an instance where the greedy policy
is strictly below P*; planted mistakes caught.
"""
import importlib.util
import random

import pytest

from oracle import online as ON
from oracle import packing as PK


def ticks(t, r, K, delta, latency, capacity):
    """Tick-by-tick simulation of the policy (small clocks only)."""
    n = len(t)
    kk = (lambda x: int(K)) if not isinstance(K, (list, tuple)) else (lambda x: int(K[x]))
    cap = capacity if capacity is not None else n + 1
    arrivals = {}
    for i in sorted(range(n), key=lambda i: (t[i], i)):
        arrivals.setdefault(t[i], []).append(i)
    queues, z = {}, [0] * n
    fb_d = fb_c = 0
    batches = []
    for tau in range(min(t), max(t) + delta + 1):
        for i in arrivals.get(tau, []):
            q = queues.setdefault(r[i], [])
            if len(q) >= cap:
                fb_c += 1
                continue
            q.append(i)
            if len(q) == cap and cap >= kk(r[i]):
                batches.append((r[i], tau, q[:]))
                queues[r[i]] = []
        for rr in sorted(queues):
            q = queues[rr]
            while q and t[q[0]] + delta - latency == tau:
                if len(q) >= kk(rr):
                    batches.append((rr, tau, q[:]))
                    queues[rr] = q = []
                else:
                    q.pop(0)
                    fb_d += 1
    for _, _, b in batches:
        for i in b:
            z[i] = 1
    return sum(z), fb_d, fb_c, sorted(batches)


def rand_instance(rng, n, R, span):
    return [rng.randrange(span) for _ in range(n)], [rng.randrange(R) for _ in range(n)]


def test_event_loop_equals_tick_simulation():
    rng = random.Random(99)
    for trial in range(400):
        R = rng.randrange(1, 4)
        t, r = rand_instance(rng, rng.randrange(1, 25), R, rng.choice([5, 15, 40]))
        K = [rng.randrange(1, 5) for _ in range(R)] if trial % 2 else rng.randrange(1, 5)
        delta = rng.randrange(0, 10)
        L = rng.randrange(0, delta + 1)
        cap = rng.choice([None, 1, 2, 3, 5, 8])
        got = ON.online_compactor(t, r, K, delta, L, cap)
        want = ticks(t, r, K, delta, L, cap)
        assert (got["accelerated"], got["fallback_deadline"], got["fallback_capacity"],
                sorted(got["batches"])) == want, (t, r, K, delta, L, cap)


def check_batches(res, t, r, K, delta, L, cap):
    kk = (lambda x: int(K)) if not isinstance(K, (list, tuple)) else (lambda x: int(K[x]))
    seen = set()
    for rr, tau, b in res["batches"]:
        assert all(r[i] == rr for i in b)
        assert len(b) >= kk(rr)
        assert cap is None or len(b) <= cap
        assert all(t[i] <= tau and tau + L <= t[i] + delta for i in b)
        assert not (seen & set(b))
        seen |= set(b)
    assert len(seen) == res["accelerated"] == sum(res["z"])
    assert res["accelerated"] + res["fallback_deadline"] + res["fallback_capacity"] == len(t)


def test_online_is_bounded_by_exact_packing():
    rng = random.Random(123)
    for trial in range(150):
        R = rng.randrange(1, 5)
        t, r = rand_instance(rng, rng.randrange(5, 200), R, rng.choice([100, 2000, 50_000]))
        K = [rng.randrange(1, 7) for _ in range(R)] if trial % 2 else rng.randrange(1, 7)
        delta = rng.randrange(1, 1000)
        L = rng.randrange(0, delta + 1)
        cap = rng.choice([None, 4, 16, 64])
        res = ON.online_compactor(t, r, K, delta, L, cap)
        check_batches(res, t, r, K, delta, L, cap)
        p_star, _ = PK.exact_packing(t, r, K, delta)
        assert res["accelerated"] <= p_star


def test_closed_forms():
    # n simultaneous events on one route, capacity c >= K: full queues launch
    # on arrival; the remainder n mod c launches at its trigger iff >= K
    for n in (1, 7, 20, 33):
        for K, c in ((1, 4), (3, 4), (5, 5), (2, 10)):
            g = n % c
            res = ON.online_compactor([9] * n, [2] * n, K, 10, 3, c)
            assert res["accelerated"] == n - (g if g < K else 0), (n, K, c)
            assert res["fallback_deadline"] == (g if g < K else 0)
    # capacity below K: nothing launches; the overflow goes to the CPU at once
    res = ON.online_compactor([0] * 10, [0] * 10, 5, 7, 0, 3)
    assert (res["accelerated"], res["fallback_capacity"], res["fallback_deadline"]) == (0, 7, 3)
    # evenly spaced releases, spacing s, delta = m s, no latency: groups of
    # m + 1 launch; the last group of n mod (m + 1) launches iff >= K
    for n, m, K in ((40, 3, 4), (41, 3, 4), (43, 3, 2), (43, 3, 4), (10, 0, 1), (12, 2, 4)):
        t = [5 * i for i in range(n)]
        g = n % (m + 1)
        want = 0 if K > m + 1 else n - (g if 0 < g < K else 0)
        assert ON.online_compactor(t, [0] * n, K, 5 * m, 0)["accelerated"] == want, (n, m, K)
    # latency equal to delta: only events released together can share a launch
    t = [0, 0, 0, 4, 4, 9, 9, 9, 9]
    assert ON.online_compactor(t, [0] * 9, 3, 6, 6)["accelerated"] == 7


def test_greedy_is_below_the_exact_packing_here():
    # launching at the oldest deadline takes {0, 5, 10}; the exact packing
    # prefers {5, 10, 12, 14}
    t = [0, 5, 10, 12, 14]
    res = ON.online_compactor(t, [0] * 5, 3, 10, 0)
    assert res["accelerated"] == 3
    assert res["batches"] == [(0, 10, [0, 1, 2])]
    assert PK.exact_packing(t, [0] * 5, 3, 10)[0] == 4
    assert ON.recovery(3, 0, 4) == 0.75
    assert ON.recovery(3, 4, 4) is None


MUTANTS = {
    "arrival_after_trigger": ("int(t[order[p]]) <= trig[0]", "int(t[order[p]]) < trig[0]"),
    "launch_above_k": ("            if len(q) >= _k(K, rr):\n", "            if len(q) > _k(K, rr):\n"),
    "no_latency": ("tau = int(t[q[0]]) + delta - latency", "tau = int(t[q[0]]) + delta"),
    "drop_newest": ("                q.pop(0)\n", "                q.pop()\n"),
    "no_capacity_launch": ("if len(q) == cap and cap >= _k(K, rr):", "if False:"),
    "capacity_off_by_one": ("if len(q) >= cap:", "if len(q) > cap:"),
    "launch_time_of_filler": ("batches.append((rr, int(t[i]), list(q)))",
                              "batches.append((rr, int(t[q[0]]), list(q)))"),
}


def _pins(mod):
    global ON
    saved = ON
    ON = mod
    try:
        test_event_loop_equals_tick_simulation()
        test_closed_forms()
        test_greedy_is_below_the_exact_packing_here()
    finally:
        ON = saved


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_online_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(ON.__file__).read()
    assert src.count(old) == 1, "anchor not found: %s" % name
    path = tmp_path / ("online_%s.py" % name)
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location("online_" + name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    with pytest.raises(AssertionError):
        _pins(mod)
