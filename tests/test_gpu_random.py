"""Seeded random shapes on the GPU against the oracle (needs an MI355X).

Every case draws W, R, the route mode, the threshold, a mix of cohort sizes
(1..256, so that sub-wavefront and multi-wavefront cohorts share bins in
arbitrary combinations), T, the padding of ld and step0, then compares the
resident chain -- over all cohorts and over ragged cohort ranges in a
shuffled order -- and the host round trip with the oracle, bit-exactly.
Two further sets aim at the pipelined three-role kernel: W 17..32 with long
chains, and W 9..16 with short and long ones.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")
N_CASES = 24


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def draw(case):
    rng = np.random.Generator(np.random.PCG64(90_000 + case))
    W = int(rng.integers(4, 65))
    R = int(rng.choice([1, 2, 5, 16, 64, 200, 256, 1000, 1024]))
    mode = wk.ROUTE_CDF if (R > 1 and rng.random() < 0.5) else wk.ROUTE_MOD
    thr = int(rng.choice([0, 1, 3277, 19661, 32768, 65535, 65536]))
    mixes = ([32, 64, 128, 256], [1, 7, 31, 32, 33, 63, 64], [65, 100, 128, 200, 256],
             list(range(1, 257)))
    kinds = mixes[int(rng.integers(0, len(mixes)))]
    sizes = [int(x) for x in rng.choice(kinds, size=int(rng.integers(1, 40)))]
    T = int(rng.choice([1, 2, 5, 8, 16, 17, 33]))
    pad = int(rng.choice([0, 0, 3, 64]))
    step0 = int(rng.choice([0, 7, 0xFFFFFFF0]))
    return W, R, mode, thr, sizes, T, pad, step0


def assert_same(got, want, what):
    for k in KEYS:
        if not np.array_equal(got[k], want[k]):
            bad = np.argwhere(got[k] != want[k])
            raise AssertionError("%s: %s differs at %d places, first %s" % (what, k, len(bad),
                                                                           tuple(bad[0])))


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_shape(orc, case):
    W, R, mode, thr, sizes, T, pad, step0 = draw(case)
    N = sum(sizes)
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=mode, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=9000 + case, ld=N + pad)
    C = inp.n_cohorts
    say("random case %d: W=%d R=%d mode=%d thr=%d C=%d N=%d T=%d pad=%d step0=%d"
        % (case, W, R, mode, thr, C, N, T, pad, step0))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    rng = np.random.Generator(np.random.PCG64(91_000 + case))
    cuts = sorted(set([0, C] + [int(x) for x in rng.integers(0, C + 1, size=3)]))
    ranges = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)]
    rng.shuffle(ranges)
    for label, mode_run, rr in (("resident", rc.RC_MODE_RESIDENT, [(0, C)]),
                                ("resident ranges", rc.RC_MODE_RESIDENT, ranges),
                                ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP, [(0, C)])):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            for cb, ce in rr:
                co.run_chain(step0, T, mode_run, cb, ce)
            got = co.download(T)
        finally:
            co.close()
        assert_same(got, want, "case %d %s" % (case, label))


def draw_two_lane(case):
    """Shapes of the pipelined three-role kernel: W 17..32, a route count
    whose full mask image fits, long chains (T > 16), launches of at most
    256 cohorts."""
    rng = np.random.Generator(np.random.PCG64(92_000 + case))
    W = int(rng.integers(17, 33))
    R = int(rng.choice([1, 3, 16, 64, 200, 256, 400]))
    mode = wk.ROUTE_CDF if (R > 1 and rng.random() < 0.5) else wk.ROUTE_MOD
    thr = int(rng.choice([0, 3277, 19661, 32768, 65536]))
    mixes = ([256], [1, 31, 32, 33, 64, 65, 100, 255, 256], list(range(1, 257)))
    kinds = mixes[int(rng.integers(0, len(mixes)))]
    sizes = [int(x) for x in rng.choice(kinds, size=int(rng.integers(1, 60)))]
    T = int(rng.choice([17, 20, 31, 32, 33, 48]))
    pad = int(rng.choice([0, 5]))
    step0 = int(rng.choice([0, 0xFFFFFFF8]))
    return W, R, mode, thr, sizes, T, pad, step0


@pytest.mark.parametrize("case", range(12))
def test_random_two_lane_long_chain(orc, case):
    W, R, mode, thr, sizes, T, pad, step0 = draw_two_lane(case)
    N = sum(sizes)
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=mode, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=9500 + case, ld=N + pad)
    C = inp.n_cohorts
    say("two-lane case %d: W=%d R=%d mode=%d thr=%d C=%d N=%d T=%d step0=%d"
        % (case, W, R, mode, thr, C, N, T, step0))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    rng = np.random.Generator(np.random.PCG64(93_000 + case))
    cuts = sorted(set([0, C] + [int(x) for x in rng.integers(0, C + 1, size=2)]))
    ranges = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)]
    rng.shuffle(ranges)
    for label, mode_run, rr in (("resident", rc.RC_MODE_RESIDENT, [(0, C)]),
                                ("resident ranges", rc.RC_MODE_RESIDENT, ranges),
                                ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP, [(0, C)])):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            for cb, ce in rr:
                co.run_chain(step0, T, mode_run, cb, ce)
            got = co.download(T)
        finally:
            co.close()
        assert_same(got, want, "two-lane case %d %s" % (case, label))


def draw_narrow_pipelined(case):
    """Shapes of the pipelined three-role kernel at WMAX = 16: W 9..16 (the B
    lanes hold words 0..7, the C lanes 8..W-1), any route count whose full
    mask image fits, short and long chains, launches of at most 256
    workgroups (or CDF routes, pipelined at any size)."""
    rng = np.random.Generator(np.random.PCG64(94_000 + case))
    W = int(rng.integers(9, 17))
    R = int(rng.choice([1, 3, 16, 64, 256, 1000]))
    mode = wk.ROUTE_CDF if (R > 1 and rng.random() < 0.5) else wk.ROUTE_MOD
    thr = int(rng.choice([0, 3277, 19661, 32768, 65536]))
    mixes = ([64], [1, 31, 32, 33, 64, 65, 100, 255, 256], list(range(1, 257)))
    kinds = mixes[int(rng.integers(0, len(mixes)))]
    sizes = [int(x) for x in rng.choice(kinds, size=int(rng.integers(1, 80)))]
    T = int(rng.choice([1, 3, 4, 5, 8, 13, 16, 33]))
    pad = int(rng.choice([0, 7]))
    step0 = int(rng.choice([0, 0xFFFFFFFD]))
    return W, R, mode, thr, sizes, T, pad, step0


@pytest.mark.parametrize("case", range(10))
def test_random_narrow_pipelined(orc, case):
    W, R, mode, thr, sizes, T, pad, step0 = draw_narrow_pipelined(case)
    N = sum(sizes)
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=mode, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=9700 + case, ld=N + pad)
    C = inp.n_cohorts
    say("narrow pipelined case %d: W=%d R=%d mode=%d thr=%d C=%d N=%d T=%d step0=%d"
        % (case, W, R, mode, thr, C, N, T, step0))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    rng = np.random.Generator(np.random.PCG64(95_000 + case))
    cuts = sorted(set([0, C] + [int(x) for x in rng.integers(0, C + 1, size=2)]))
    ranges = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)]
    rng.shuffle(ranges)
    for label, mode_run, rr in (("resident", rc.RC_MODE_RESIDENT, [(0, C)]),
                                ("resident ranges", rc.RC_MODE_RESIDENT, ranges),
                                ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP, [(0, C)])):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            for cb, ce in rr:
                co.run_chain(step0, T, mode_run, cb, ce)
            got = co.download(T)
        finally:
            co.close()
        assert_same(got, want, "narrow pipelined case %d %s" % (case, label))
