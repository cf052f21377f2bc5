"""Route keys at their boundaries (needs an MI355X).

CDF mode on degenerate threshold sets, and MOD mode at multiples of R.

The route is the number of thresholds at or below the outcome.  The kernels
find it with a guide table and a fixed-trip binary search (the resident
chain) or a search over the thresholds (the host-round-trip body).  Here the
thresholds repeat, sit at 0 and 2^32 - 1, crowd into one guide bucket, or are
all equal.  The step-0 outcomes are inputs, so sessions are given outcomes
on and next to every threshold.  Every shape runs through the non-split
chain (W = 8), the split or table-image chain (W = 32) and the table image
(W = 64, R = 1024), in both mechanisms, against the oracle bit for bit.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")
M32 = 0xFFFFFFFF


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def cdf_of(name):
    rng = np.random.Generator(np.random.PCG64(34_000))
    if name == "ties and extremes":
        return np.asarray([0, 0, 5, 5, 5, M32], dtype=np.uint32)
    if name == "one bucket":
        return np.asarray([1, 0x100], dtype=np.uint32)
    if name == "clustered":
        return np.sort((1 << 31) + rng.integers(0, 4096, size=1023)).astype(np.uint32)
    if name == "all at the top":
        return np.full(1023, M32, dtype=np.uint32)
    if name == "all at zero":
        return np.zeros(1023, dtype=np.uint32)
    return wk.zipf_cdf(1024, 1.1)


CDFS = ["ties and extremes", "one bucket", "clustered", "all at the top", "all at zero", "zipf"]


def boundary_outcomes(cdf):
    vals = {0, 1, M32 - 1, M32}
    for v in np.unique(cdf).tolist():
        vals.update({(v - 1) & M32, v, (v + 1) & M32})
    return np.asarray(sorted(vals), dtype=np.uint32)


@pytest.mark.parametrize("W", [8, 32, 64])
@pytest.mark.parametrize("name", CDFS)
def test_degenerate_cdf(orc, name, W):
    cdf = cdf_of(name)
    R = cdf.size + 1
    sizes = [256, 64, 1, 31, 100, 256, 200, 7, 128] * 2
    T, thr, step0 = 3, 19661, 11
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=wk.ROUTE_CDF, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=34_000 + W, route_cdf=cdf,
                         ld=sum(sizes) + 5)
    edges = boundary_outcomes(cdf)
    N = inp.n_sessions
    n_edge = min(N, max(2 * edges.size, N // 4))
    pos = np.random.Generator(np.random.PCG64(34_001)).permutation(N)[:n_edge]
    inp.outcome[pos] = np.resize(edges, pos.size)
    say("cdf %s: R=%d W=%d C=%d N=%d boundary outcomes=%d" % (name, R, W, inp.n_cohorts, N,
                                                            pos.size))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    for label, mode in (("resident", rc.RC_MODE_RESIDENT),
                        ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP)):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            co.run_chain(step0, T, mode)
            got = co.download(T)
        finally:
            co.close()
        for k in KEYS:
            assert np.array_equal(got[k], want[k]), (name, W, label, k)


def mod_boundary_outcomes(R):
    top = (M32 // R) * R
    vals = {0, 1, M32 - 1, M32, top, (top - 1) & M32, top + 1 if top < M32 else 0}
    for k in (1, 2, 3, 1000, 65535, 1 << 20):
        if k * R <= M32:
            vals.update({k * R - 1, k * R, (k * R + 1) & M32})
    return np.asarray(sorted(vals), dtype=np.uint32)


@pytest.mark.parametrize("W", [8, 32, 64])
@pytest.mark.parametrize("R", [1, 3, 7, 1000, 1023, 1024])
def test_mod_boundaries(orc, R, W):
    """MOD route mode, step-0 outcomes on and next to multiples of R and at
    the top of the u32 range (power-of-two R takes the masked form)."""
    sizes = [256, 64, 1, 31, 100, 256, 200, 7, 128] * 2
    T, thr, step0 = 3, 32768, 0
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=wk.ROUTE_MOD, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=35_000 + W + R)
    edges = mod_boundary_outcomes(R)
    N = inp.n_sessions
    pos = np.random.Generator(np.random.PCG64(35_001)).permutation(N)[:N // 4]
    inp.outcome[pos] = np.resize(edges, pos.size)
    say("mod R=%d W=%d C=%d N=%d boundary outcomes=%d" % (R, W, inp.n_cohorts, N, pos.size))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    for label, mode in (("resident", rc.RC_MODE_RESIDENT),
                        ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP)):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            co.run_chain(step0, T, mode)
            got = co.download(T)
        finally:
            co.close()
        for k in KEYS:
            assert np.array_equal(got[k], want[k]), (R, W, label, k)
