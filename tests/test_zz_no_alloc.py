"""The entry point that allocates nothing, rc_cohort_run_chain_noalloc
(needs an MI355X).

It is rc_cohort_run_chain with the host round trip's scratch in the
library's fixed device array.  Its outputs must equal rc_cohort_run_chain's
on the same inputs bit for bit (both are checked against the oracle too), on
two calls in a row of which the second has the smaller input, in both
mechanisms; a chain continued by it on a second stream must wait for the
first call; at the session limit it runs, and beyond it the call is refused
before anything is enqueued.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")
MODES = {"resident": rc.RC_MODE_RESIDENT, "host_rt": rc.RC_MODE_HOST_ROUNDTRIP}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def run_both(inp, T, mode, cb=0, ce=None, step0=0):
    """(run_chain outputs, run_chain_noalloc outputs) on fresh buffers."""
    out = []
    for entry in ("run_chain", "run_chain_noalloc"):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            ce_ = co.n_cohorts if ce is None else ce
            fn = getattr(rc, "rc_cohort_" + entry)
            fn(co.handle, co.buffers, step0, T, mode, cb, ce_, None)
            out.append(co.download(T))
        finally:
            co.close()
    return out


# first call: a larger input; second call: a smaller one (another handle,
# fewer sessions and words), so the second reuses a smaller part of the array
CALLS = [
    dict(n_words=32, n_routes=64, route_mode=wk.ROUTE_CDF, decide_thr=19661,
         cohort_sizes=[256] * 60 + [17, 100, 64, 31], n_steps=6, seed_key=77_001),
    dict(n_words=16, n_routes=16, route_mode=wk.ROUTE_MOD, decide_thr=32768,
         cohort_sizes=[64, 32, 5, 64], n_steps=3, seed_key=77_002),
]


@pytest.mark.parametrize("mode", sorted(MODES))
def test_noalloc_equals_run_chain_two_calls(orc, mode):
    for i, kw in enumerate(CALLS):
        inp = wk.make_custom(**kw)
        T = kw["n_steps"]
        say("noalloc %s call %d: W=%d N=%d T=%d" % (mode, i, inp.n_words, inp.n_sessions, T))
        ref, got = run_both(inp, T, MODES[mode], step0=3 + i)
        want = orc.run_inputs(inp, n_steps=T, step0=3 + i)
        for k in KEYS:
            assert np.array_equal(got[k], ref[k]), (mode, i, k)
            assert np.array_equal(got[k], want[k]), (mode, i, k)


def test_noalloc_counts(orc):
    inp = wk.make_custom(**CALLS[1])
    co = rc.Cohort.from_inputs(inp, max_steps=3)
    try:
        co.run_chain_noalloc(0, 3, rc.RC_MODE_HOST_ROUNDTRIP)
        launches, copies = co.last_counts()
        assert copies == 3 and launches >= 3 + 1 + 1  # decides, bodies, the counter clear
        co.run_chain_noalloc(0, 3, rc.RC_MODE_RESIDENT)
        assert co.last_counts() == (1, 0)
    finally:
        co.close()


def test_noalloc_two_streams(orc):
    import test_gpu_streams
    test_gpu_streams.one_handle_two_streams(orc, "run_chain_noalloc")


def test_noalloc_session_limit(orc):
    """A range of exactly RC_NOALLOC_MAX_SESSIONS sessions runs (host round
    trip, one step, against run_chain); one more session is refused with
    RC_E_INVALID before any launch, and the outputs stay untouched."""
    lim = rc.RC_NOALLOC_MAX_SESSIONS
    sizes = [256] * (lim // 256) + [1]
    inp = wk.make_custom(n_words=4, n_routes=8, route_mode=wk.ROUTE_MOD, decide_thr=32768,
                         cohort_sizes=sizes, n_steps=1, seed_key=77_003)
    C = inp.n_cohorts
    say("noalloc limit: N=%d C=%d" % (inp.n_sessions, C))
    ref, got = run_both(inp, 1, rc.RC_MODE_HOST_ROUNDTRIP, cb=0, ce=C - 1)
    for k in KEYS:
        assert np.array_equal(got[k], ref[k]), k
    co = rc.Cohort.from_inputs(inp, max_steps=1)
    try:
        before = co.download(1)
        st = rc.rc_cohort_run_chain_noalloc(co.handle, co.buffers, 0, 1, rc.RC_MODE_HOST_ROUNDTRIP,
                                            0, C, None, check=False)
        assert st == rc.RC_E_INVALID
        after = co.download(1)
        for k in KEYS:
            assert np.array_equal(before[k], after[k]), k
    finally:
        co.close()
