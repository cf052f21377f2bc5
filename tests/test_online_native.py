"""The library's online route compactor (``rc_online_compact``) and cohort
builder (``rc_cohorts_from_batches``), host code, against the oracle.

The frozen policy is deterministic, so the native result must equal the
oracle's exactly: the counts, and every batch (route, launch time, members).
On the 1M-event arrival stream the oracle runs sampled routes whole, and
every batch of every route is checked for feasibility; A <= P* against the
library's own exact packing there.
"""
import random

import numpy as np
import pytest

from oracle import online as ON
from oracle import packing as PK
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

NONE = 0xFFFFFFFF


def native(t, r, K, delta, L, cap, n_routes):
    k = np.full(n_routes, K, dtype=np.uint32) if np.isscalar(K) else np.asarray(K, dtype=np.uint32)
    return rc.rc_online_compact(release_ns=np.asarray(t, dtype=np.int64),
                                route=np.asarray(r, dtype=np.uint32), k_of_route=k,
                                delta_ns=delta, latency_ns=L,
                                capacity=rc.UNLIMITED if cap is None else cap, witness=True)


def batch_sets(bat, lt, r):
    out = []
    for b in range(lt.size):
        m = np.flatnonzero(bat == b)
        out.append((int(r[m[0]]), int(lt[b]), sorted(int(i) for i in m)))
    return sorted(out)


def compare(t, r, K, delta, L, cap, n_routes):
    res, bat, lt = native(t, r, K, delta, L, cap, n_routes)
    kd = K if np.isscalar(K) else list(K)
    want = ON.online_compactor(list(t), list(r), kd, delta, L, cap)
    got = (res["accelerated"], res["fallback_deadline"], res["fallback_capacity"],
           res["n_batches"])
    assert got == (want["accelerated"], want["fallback_deadline"], want["fallback_capacity"],
                   len(want["batches"])), (got, t, r, K, delta, L, cap)
    wb = sorted((rr, tau, sorted(b)) for rr, tau, b in want["batches"])
    assert batch_sets(bat, lt, np.asarray(r)) == wb
    at_cap = sum(1 for _, _, b in want["batches"] if cap is not None and len(b) == cap)
    assert res["launched_at_capacity"] == at_cap
    # numbering: by route, then launch order
    keys = [(int(np.asarray(r)[np.flatnonzero(bat == b)[0]]), int(lt[b])) for b in range(lt.size)]
    assert keys == sorted(keys)
    return res, bat, lt


def test_random_instances_match_the_oracle():
    rng = random.Random(31337)
    for trial in range(400):
        R = rng.randrange(1, 6)
        n = rng.randrange(1, 160)
        span = rng.choice([10, 300, 20_000])
        t = [rng.randrange(-span, span) for _ in range(n)]
        r = [rng.randrange(R) for _ in range(n)]
        K = [rng.randrange(1, 8) for _ in range(R)] if trial % 3 else rng.randrange(1, 8)
        delta = rng.choice([0, 1, rng.randrange(1, 60), rng.randrange(1, span + 1)])
        L = rng.choice([0, delta, rng.randrange(0, delta + 1)])
        cap = rng.choice([None, 1, 2, 5, 16, 64])
        if delta == 0:
            delta = 1
            L = min(L, 1)
        compare(t, r, K, delta, L, cap, R)


def test_degenerate_inputs():
    res, bat, lt = native([], [], 2, 10, 0, None, 3)
    assert res["accelerated"] == res["n_batches"] == 0 and lt.size == 0
    # capacity below K: nothing ever launches
    res, _, _ = compare([0] * 10, [0] * 10, 5, 7, 0, 3, 1)
    assert (res["accelerated"], res["fallback_capacity"], res["fallback_deadline"]) == (0, 7, 3)
    # latency = delta
    compare([0, 0, 0, 4, 4, 9, 9, 9, 9], [0] * 9, 3, 6, 6, None, 1)
    big = (2 ** 63 - 1) // 4
    compare([big, big - 1, -big, -big + 2], [0, 0, 1, 1], 2, 3, 1, None, 2)


def test_invalid_arguments():
    t = np.array([0, 1], dtype=np.int64)
    r = np.array([0, 1], dtype=np.uint32)
    k = np.array([1, 1], dtype=np.uint32)

    def st(**kw):
        args = dict(release_ns=t, route=r, k_of_route=k, delta_ns=5)
        args.update(kw)
        return rc.rc_online_compact(check=False, **args)

    assert isinstance(st(), dict)
    assert st(latency_ns=6) == rc.RC_E_INVALID
    assert st(latency_ns=-1) == rc.RC_E_INVALID
    assert st(capacity=0) == rc.RC_E_INVALID
    assert st(route=np.array([0, 5], dtype=np.uint32)) == rc.RC_E_INVALID
    assert st(k_of_route=np.array([0, 1], dtype=np.uint32)) == rc.RC_E_INVALID
    assert st(delta_ns=0, latency_ns=0) == rc.RC_E_INVALID
    # cohort builder
    b = np.array([0, NONE, 1, 0], dtype=np.uint32)
    assert rc.rc_cohorts_from_batches(b, 1, check=False) == rc.RC_E_INVALID  # id 1 >= 1
    assert rc.rc_cohorts_from_batches(b, 2, max_cohort=0, check=False) == rc.RC_E_INVALID
    assert rc.rc_cohorts_from_batches(b, 5, check=False) == rc.RC_E_INVALID  # n_batches > n
    with pytest.raises(rc.RcError):
        rc.rc_cohorts_from_batches(b, 1)


def test_cohorts_from_batches_layout():
    b = np.array([1, 0, NONE, 1, 0, 1, 1, 1, NONE, 0], dtype=np.uint32)
    order, off = rc.rc_cohorts_from_batches(b, 2, max_cohort=2)
    # batch 0 = events 1, 4, 9 -> cohorts [1, 4], [9]; batch 1 = 0, 3, 5, 6, 7 -> [0, 3], [5, 6], [7]
    assert order.tolist() == [1, 4, 9, 0, 3, 5, 6, 7]
    assert off.tolist() == [0, 2, 3, 5, 7, 8]
    rng = np.random.default_rng(8)
    for _ in range(30):
        n = int(rng.integers(1, 3000))
        nb = int(rng.integers(1, 40))
        b = rng.integers(0, nb, n).astype(np.uint32)
        b[rng.random(n) < 0.2] = NONE
        mc = int(rng.choice([1, 7, 32, 256]))
        order, off = rc.rc_cohorts_from_batches(b, nb, max_cohort=mc)
        kept = np.flatnonzero(b != NONE)
        assert sorted(order.tolist()) == kept.tolist()
        sizes = np.diff(off)
        assert (sizes >= 1).all() and (sizes <= mc).all()
        for c in range(sizes.size):
            m = order[off[c]:off[c + 1]]
            assert np.unique(b[m]).size == 1           # one batch per cohort
            assert (np.diff(m.astype(np.int64)) > 0).all()  # index order
        # near-equal pieces: per batch the sizes differ by at most one and
        # their count is ceil(n_b / max)
        cb = b[order[off[:-1]]]
        for bb in np.unique(cb):
            s = sizes[cb == bb]
            nbb = int((b == bb).sum())
            assert s.size == -(-nbb // mc) and s.max() - s.min() <= 1 and s.sum() == nbb


@pytest.fixture(scope="module")
def arrivals():
    wl = wk.WORKLOADS["s1m"]
    times, routes, _ = wk.arrival_events(wl)
    return wl, times, routes


@pytest.mark.parametrize("K,L,cap", [(32, 25_000, 4096), (256, 25_000, 256), (64, 0, rc.UNLIMITED)])
def test_arrival_stream(arrivals, K, L, cap):
    wl, times, routes = arrivals
    R = wl.n_routes
    k = np.full(R, K, dtype=np.uint32)
    delta = wk.DEADLINE_NS
    res, bat, lt = rc.rc_online_compact(release_ns=times, route=routes, k_of_route=k,
                                        delta_ns=delta, latency_ns=L, capacity=cap, witness=True)
    n = times.size
    assert res["accelerated"] + res["fallback_deadline"] + res["fallback_capacity"] == n
    assert int((bat != NONE).sum()) == res["accelerated"]
    packed = rc.rc_pack_shares(release_ns=times, route=routes, k_of_route=k, delta_ns=delta)
    assert res["accelerated"] <= packed["packed"]
    # every batch feasible with the latency: t_j <= tau, tau + L <= t_j + delta
    m = bat != NONE
    b = bat[m].astype(np.int64)
    tj = times[m]
    assert (tj <= lt[b]).all() and (lt[b] + L <= tj + delta).all()
    sizes = np.bincount(b, minlength=lt.size)
    assert (sizes >= K).all() and (sizes <= min(cap, n)).all()
    # sampled routes through the oracle, whole
    counts = np.bincount(routes, minlength=R)
    rng = np.random.default_rng(K)
    for rr in rng.choice(np.flatnonzero((counts > 50) & (counts < 1500)), 4, replace=False):
        sel = np.flatnonzero(routes == rr)
        compare(times[sel].tolist(), [0] * sel.size, K, delta, L, None if cap == rc.UNLIMITED else cap, 1)
