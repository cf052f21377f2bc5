"""Every invocation of the two per-cohort chained workloads, in both
mechanisms, bit-exact against the oracle (needs an MI355X).

The K = 64 workload is 10,000 invocations (10 descriptors of 1,000 cohorts)
and the K = 256 workload 50,000 (50 descriptors of 1,000); an invocation is
one run_chain call over a single cohort, step numbers from 0.  Each
descriptor's outputs -- final state, next outcomes, every effect slice and
every count -- are compared whole with the oracle's, after the resident
chain and again after the host round trip on fresh buffers.  The oracle runs
on disjoint cohort ranges in host threads, all writing into one set of
output arrays (each call touches only its own cohorts' sessions, slots and
counts).
"""
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")
THREADS = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def oracle_threaded(orc, inp, T):
    C, ld = inp.n_cohorts, inp.ld
    state, outcome = inp.state.copy(), inp.outcome.copy()
    fill = np.uint32(0xFFFFFFFF)
    out = dict(eff_sid=np.full((T, ld), fill, dtype=np.uint32),
               eff_tool=np.full((T, ld), fill, dtype=np.uint32),
               eff_payload=np.full((T, ld, 4), fill, dtype=np.uint32),
               n_taken=np.full((T, C), fill, dtype=np.uint32))
    cuts = [C * i // THREADS for i in range(THREADS + 1)]

    def part(i):
        orc.run_chain(n_words=inp.n_words, n_routes=inp.n_routes, cohort_offsets=inp.cohort_offsets,
                      table=inp.table, route_mode=inp.route_mode, route_cdf=inp.route_cdf,
                      decide_thr=inp.decide_thr, state=state, outcome=outcome, n_steps=T,
                      cohort_begin=cuts[i], cohort_end=cuts[i + 1], **out)

    with ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(part, [i for i in range(THREADS) if cuts[i] < cuts[i + 1]]))
    return dict(state=state, outcome=outcome, **out)


CHUNKS = [("k64", c) for c in range(wk.n_chunks(wk.WORKLOADS["k64"]))] + \
         [("k256", c) for c in range(wk.n_chunks(wk.WORKLOADS["k256"]))]


@pytest.mark.parametrize("key,chunk", CHUNKS)
def test_every_invocation(orc, key, chunk):
    wl = wk.WORKLOADS[key]
    T = wl.n_steps
    inp = wk.make_inputs(wl, chunk=chunk)
    say("%s chunk %d: %d invocations, T=%d" % (key, chunk, inp.n_cohorts, T))
    want = oracle_threaded(orc, inp, T)
    for mode in (rc.RC_MODE_RESIDENT, rc.RC_MODE_HOST_ROUNDTRIP):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            for c in range(inp.n_cohorts):
                co.run_chain(0, T, mode, c, c + 1)
            got = co.download(T)
        finally:
            co.close()
        for k in KEYS:
            if not np.array_equal(got[k], want[k]):
                bad = np.argwhere(got[k] != want[k])
                raise AssertionError("%s chunk %d mode %d: %s differs at %d places, first %s"
                                     % (key, chunk, mode, k, len(bad), tuple(bad[0])))
