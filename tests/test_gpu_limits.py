"""The HIP path at the descriptor's size limits (needs an MI355X).

Two corners that the other parity tests do not reach:
- the largest leading dimension, ld = RC_MAX_SESSIONS = 2^28, with a few
  thousand sessions: word rows and effect slices lie gigabytes apart, so the
  kernels' 64-bit address arithmetic is exercised.  W = 64 (table image),
  W = 32 (split full image) and W = 4, in both mechanisms and the floor; the
  padding columns [N, ld) of every buffer must come back untouched;
- the largest session count, N = 2^28 (1,048,578 cohorts, a ragged tail):
  sampled cohorts against the oracle, every effect slice checked to hold, at
  each slot, a session of the slot's cohort and all N sessions once, and the
  host round trip equal to the resident chain over every output;
- the largest LDS footprint of a chain workgroup: the full mask image, which
  every W <= 16 takes, with about a thousand CDF routes and their guide table
  of 2^12 buckets -- about 146 KB of LDS per workgroup, one workgroup per CU,
  the pipelined split -- against the oracle bit for bit, in both mechanisms
  and over ragged cohort ranges.
The first uses 77 GiB of device memory at W = 64, the second about 45 GiB.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")
FILL = -1  # 0xFFFFFFFF, the fill of every output buffer


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def host(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32).copy()


def untouched(t) -> bool:
    return int(t.min()) == FILL and int(t.max()) == FILL


def assert_same(got, want, what):
    for k in KEYS:
        g, w = got[k], want[k]
        assert g.shape == w.shape, (what, k, g.shape, w.shape)
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            raise AssertionError("%s: %s differs at %d places, first %s" % (what, k, len(bad),
                                                                           tuple(bad[0])))


def release(*cohorts):
    import torch
    for co in cohorts:
        co.close()
        co.t.clear()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# (W, R, route mode, thr, cohort sizes)
LD_CASES = {
    "table image": (64, 1024, wk.ROUTE_CDF, 3277, [256, 31, 32, 100, 1, 64, 200, 128, 77] * 3),
    "split image": (32, 256, wk.ROUTE_MOD, 32768, [256] * 9 + [160]),
    "narrow": (4, 16, wk.ROUTE_MOD, 19661, [32, 1, 255, 64, 17] * 4),
}


@pytest.mark.parametrize("case", sorted(LD_CASES))
def test_largest_leading_dimension(orc, case):
    import torch
    W, R, mode, thr, sizes = LD_CASES[case]
    T, step0, ld = 2, 0xFFFFFFFF, rc.RC_MAX_SESSIONS
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=mode, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=31_000 + W)
    N = inp.n_sessions
    say("largest ld, %s: W=%d R=%d mode=%d C=%d N=%d ld=%d T=%d step0=%#x"
        % (case, W, R, mode, inp.n_cohorts, N, ld, T, step0))
    want = orc.run_inputs(inp, n_steps=T, step0=step0, record=True)
    bits = np.zeros((T, (ld + 31) // 32), dtype=np.uint32)
    bits[:, :want["decisions"].shape[1]] = want["decisions"]

    co = rc.Cohort(n_words=W, n_routes=R, cohort_offsets=inp.cohort_offsets, table=inp.table,
                   route_mode=mode, route_cdf=inp.route_cdf, decide_thr=thr, max_steps=T, ld=ld)
    try:
        st0 = torch.from_numpy(inp.state.view(np.int32)).to(co.device)
        oc0 = torch.from_numpy(inp.outcome.view(np.int32)).to(co.device)
        for label in ("resident", "host round trip", "floor"):
            say("  " + label)
            for k in ("eff_sid", "eff_tool", "eff_payload", "n_taken"):
                co.t[k].fill_(FILL)
            co.t["state"][:, :N].copy_(st0)
            co.t["outcome"][:N].copy_(oc0)
            if label == "floor":
                co.run_floor(bits, T)
            else:
                co.run_chain(step0, T, rc.RC_MODE_RESIDENT if label == "resident"
                             else rc.RC_MODE_HOST_ROUNDTRIP)
            torch.cuda.synchronize()
            got = {"state": host(co.t["state"][:, :N]), "outcome": host(co.t["outcome"][:N]),
                   "eff_sid": host(co.t["eff_sid"][:, :N]),
                   "eff_tool": host(co.t["eff_tool"][:, :N]),
                   "eff_payload": host(co.t["eff_payload"][:, :N]),
                   "n_taken": host(co.t["n_taken"])}
            assert_same(got, want, "%s %s" % (case, label))
            for k in ("state", "eff_sid", "eff_tool", "eff_payload"):
                assert untouched(co.t[k][:, N:]), (case, label, k, "padding columns written")
            assert untouched(co.t["outcome"][N:]), (case, label, "outcome padding written")
    finally:
        release(co)


def test_largest_session_count(orc):
    import torch
    N = rc.RC_MAX_SESSIONS
    tail = [200, 37, 19]
    sizes = np.concatenate([np.full((N - sum(tail)) // 256, 256, dtype=np.int64), tail])
    assert int(sizes.sum()) == N
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint32)
    C = offsets.size - 1
    W, R, mode, thr, T, step0 = 4, 1024, wk.ROUTE_CDF, 19661, 2, 0xFFFFFFFF
    table = wk.uniform_u32(R * 16, 32_000, 1).reshape(R, 16)
    cdf = wk.zipf_cdf(R, 1.1)
    say("largest N: W=%d R=%d CDF C=%d N=%d T=%d step0=%#x" % (W, R, C, N, T, step0))
    mk = lambda: rc.Cohort(n_words=W, n_routes=R, cohort_offsets=offsets, table=table,
                           route_mode=mode, route_cdf=cdf, decide_thr=thr, max_steps=T)
    co = mk()
    co2 = None
    try:
        dev = co.device
        co.t["state"].copy_(wk.device_uniform_u32((W, N), 32_000, 2, device=dev))
        co.t["outcome"].copy_(wk.device_uniform_u32((N,), 32_000, 3, device=dev))
        st_in, oc_in = co.t["state"].clone(), co.t["outcome"].clone()
        rng = np.random.Generator(np.random.PCG64(32_000))
        starts = [0, C - 6] + sorted(int(x) for x in rng.integers(1, C - 12, size=6))
        samples = {(cb, cb + 6): None for cb in starts}
        for cb, ce in samples:
            b, e = int(offsets[cb]), int(offsets[ce])
            samples[(cb, ce)] = (host(co.t["state"][:, b:e]), host(co.t["outcome"][b:e]))

        say("  resident")
        co.run_chain(step0, T, rc.RC_MODE_RESIDENT)
        torch.cuda.synchronize()
        for (cb, ce), (st, oc) in samples.items():
            b, e = int(offsets[cb]), int(offsets[ce])
            want = orc.run_chain(n_words=W, n_routes=R, cohort_offsets=offsets[cb:ce + 1] - b,
                                 table=table, route_mode=mode, route_cdf=cdf, decide_thr=thr,
                                 state=st, outcome=oc, n_steps=T, step0=step0)
            got = {"state": host(co.t["state"][:, b:e]), "outcome": host(co.t["outcome"][b:e]),
                   "eff_sid": host(co.t["eff_sid"][:, b:e]) - np.uint32(b),
                   "eff_tool": host(co.t["eff_tool"][:, b:e]),
                   "eff_payload": host(co.t["eff_payload"][:, b:e]),
                   "n_taken": host(co.t["n_taken"][:, cb:ce])}
            assert_same(got, want, "largest N, cohorts [%d, %d)" % (cb, ce))

        say("  effect slices: within-cohort permutations")
        ends = torch.from_numpy(offsets[1:].astype(np.int64)).to(dev)
        slots = torch.arange(N, dtype=torch.int64, device=dev)
        cohort_of_slot = torch.searchsorted(ends, slots, right=True)
        for t in range(T):
            sid = co.t["eff_sid"][t].to(torch.int64)
            assert torch.equal(torch.searchsorted(ends, sid, right=True), cohort_of_slot), t
            assert torch.equal(torch.sort(sid).values, slots), t
        del sid, slots, cohort_of_slot

        say("  host round trip")
        co2 = mk()
        co2.t["state"].copy_(st_in)
        co2.t["outcome"].copy_(oc_in)
        del st_in, oc_in
        co2.run_chain(step0, T, rc.RC_MODE_HOST_ROUNDTRIP)
        torch.cuda.synchronize()
        for k in KEYS:
            assert torch.equal(co2.t[k], co.t[k]), k
    finally:
        release(*(c for c in (co, co2) if c is not None))


# (W, R, T, step0): full mask image at W <= 16 with ~1,000 CDF routes
LDS_CASES = [(16, 1024, 9, 0), (13, 1000, 20, 0xFFFFFFF9), (9, 1024, 4, 77)]


@pytest.mark.parametrize("case", range(len(LDS_CASES)))
def test_largest_lds_footprint(orc, case):
    W, R, T, step0 = LDS_CASES[case]
    rng = np.random.Generator(np.random.PCG64(36_000 + case))
    sizes = [int(x) for x in rng.choice([1, 17, 32, 63, 64, 65, 128, 200, 256], size=300)]
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=wk.ROUTE_CDF, decide_thr=19661,
                         cohort_sizes=sizes, n_steps=T, seed_key=36_100 + case)
    C = inp.n_cohorts
    say("largest LDS footprint: W=%d R=%d CDF C=%d N=%d T=%d step0=%d"
        % (W, R, C, inp.n_sessions, T, step0))
    want = orc.run_inputs(inp, n_steps=T, step0=step0)
    cuts = sorted(set([0, C] + [int(x) for x in rng.integers(0, C + 1, size=3)]))
    ranges = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)]
    rng.shuffle(ranges)
    for label, mode, rr in (("resident", rc.RC_MODE_RESIDENT, [(0, C)]),
                            ("resident ranges", rc.RC_MODE_RESIDENT, ranges),
                            ("host round trip", rc.RC_MODE_HOST_ROUNDTRIP, [(0, C)])):
        co = rc.Cohort.from_inputs(inp, max_steps=T)
        try:
            for cb, ce in rr:
                co.run_chain(step0, T, mode, cb, ce)
            got = co.download(T)
        finally:
            co.close()
        for k in KEYS:
            assert np.array_equal(got[k], want[k]), (case, label, k)
