"""Cohorts formed by the library's former and online compactor, fed to the
resident chain on the GPU (needs an MI355X), bit-exact against the oracle.

The 1M-event Poisson arrival stream (Zipf routes over R = 1024, delta =
50 ms) is cut into batches by the exact packing witness (rc_pack_shares) or
by the online policy (rc_online_compact); rc_cohorts_from_batches turns the
batches into cohorts of at most 256 sessions, each session starting from its
arrival's outcome; the chain then runs T = 16 steps with the 1M workload's
shape (W = 64, p = 0.05).
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


@pytest.fixture(scope="module")
def stream():
    wl = wk.WORKLOADS["s1m"]
    times, routes, outcomes = wk.arrival_events(wl)
    return wl, times, routes, outcomes


def feed_inputs(wl, routes, outcomes, bat, n_batches, seed_key):
    order, off = rc.rc_cohorts_from_batches(bat, n_batches, max_cohort=256)
    sizes = np.diff(off)
    # a cohort is one route: the route every session starts from
    first = routes[order[off[:-1]]]
    assert np.array_equal(np.repeat(first, sizes), routes[order])
    inp = wk.make_custom(n_words=wl.n_words, n_routes=wl.n_routes, route_mode=wl.route_mode,
                         decide_thr=wl.decide_thr, cohort_sizes=sizes, n_steps=wl.n_steps,
                         zipf_s=wl.zipf_s, seed_key=seed_key)
    inp.outcome[:order.size] = outcomes[order]
    return inp


def run_and_compare(orc, inp, what):
    T = inp.n_steps
    say("feed %s: N=%d C=%d T=%d" % (what, inp.n_sessions, inp.n_cohorts, T))
    want = orc.run_inputs(inp, n_steps=T)
    co = rc.Cohort.from_inputs(inp, max_steps=T)
    try:
        co.run_chain(0, T)
        got = co.download(T)
    finally:
        co.close()
    for k in KEYS:
        if not np.array_equal(got[k], want[k]):
            bad = np.argwhere(got[k] != want[k])
            raise AssertionError("%s: %s differs at %d places, first %s" % (what, k, len(bad),
                                                                           tuple(bad[0])))


@pytest.mark.parametrize("K", [32, 256])
def test_exact_packing_cohorts_on_the_chain(orc, stream, K):
    wl, times, routes, outcomes = stream
    k = np.full(wl.n_routes, K, dtype=np.uint32)
    res, bat = rc.rc_pack_shares(release_ns=times, route=routes, k_of_route=k,
                                 delta_ns=wk.DEADLINE_NS, witness=True)
    inp = feed_inputs(wl, routes, outcomes, bat, res["n_batches"], 700 + K)
    assert inp.n_sessions == res["packed"]
    run_and_compare(orc, inp, "exact packing K=%d" % K)


@pytest.mark.parametrize("K,cap", [(32, 4096), (128, 256)])
def test_online_cohorts_on_the_chain(orc, stream, K, cap):
    wl, times, routes, outcomes = stream
    k = np.full(wl.n_routes, K, dtype=np.uint32)
    res, bat, _ = rc.rc_online_compact(release_ns=times, route=routes, k_of_route=k,
                                       delta_ns=wk.DEADLINE_NS, latency_ns=25_000, capacity=cap,
                                       witness=True)
    inp = feed_inputs(wl, routes, outcomes, bat, res["n_batches"], 800 + K)
    assert inp.n_sessions == res["accelerated"]
    run_and_compare(orc, inp, "online K=%d cap=%d" % (K, cap))
