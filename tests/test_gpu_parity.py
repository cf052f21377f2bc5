"""Bit-exact parity of the HIP path with the oracle (needs an MI355X).

Every comparison is of whole output arrays: state (including the poisoned
padding columns), next outcomes, every effect slice (slots never written keep
the 0xFFFFFFFF fill on both sides) and every per-cohort count.  Both
mechanisms -- device-resident chain and host round trip -- are checked.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12123_amd import rc_cohort as rc
from paper_2608_12123_amd import workload as wk

pytestmark = pytest.mark.gpu

MODES = {"resident": rc.RC_MODE_RESIDENT, "host_rt": rc.RC_MODE_HOST_ROUNDTRIP}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


def assert_same(got, want, what=""):
    for k in ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken"):
        g, w = got[k], want[k]
        assert g.shape == w.shape, (what, k, g.shape, w.shape)
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            raise AssertionError("%s: %s differs at %d places, first %s: gpu %#x oracle %#x"
                                 % (what, k, len(bad), tuple(bad[0]), int(g[tuple(bad[0])]),
                                    int(w[tuple(bad[0])])))


def oracle_run(orc, inp, n_steps, step0=0, cb=0, ce=None):
    return orc.run_inputs(inp, n_steps=n_steps, step0=step0, cohort_begin=cb, cohort_end=ce)


def gpu_run_ranges(inp, n_steps, mode, ranges, step0=0):
    """One run_chain call per cohort range (an 'invocation')."""
    co = rc.Cohort.from_inputs(inp, max_steps=max(n_steps, 1))
    try:
        for cb, ce in ranges:
            co.run_chain(step0, n_steps, mode, cb, ce)
        return co.download(n_steps)
    finally:
        co.close()


# ---------------------------------------------------------------------------
# the five benchmark workloads
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("key,n_inv", [("tiny", 1000), ("k64", 1000), ("k256", 120)])
def test_per_cohort_workload(orc, key, n_inv, mode):
    """Independent invocations, one cohort each, step numbers from 0."""
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl, chunk=0)
    say("case %s mode=%s invocations=%d T=%d W=%d R=%d" % (key, mode, n_inv, wl.n_steps,
                                                          wl.n_words, wl.n_routes))
    ranges = [(c, c + 1) for c in range(n_inv)]
    got = gpu_run_ranges(inp, wl.n_steps, MODES[mode], ranges)
    want = oracle_run(orc, inp, wl.n_steps, cb=0, ce=n_inv)
    assert_same(got, want, key)


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("key", ["s100k", "s1m"])
def test_single_launch_workload(orc, key, mode):
    """The whole workload in one call, at full size."""
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl)
    say("case %s mode=%s N=%d C=%d T=%d" % (key, mode, inp.n_sessions, inp.n_cohorts, wl.n_steps))
    got = gpu_run_ranges(inp, wl.n_steps, MODES[mode], [(0, inp.n_cohorts)])
    want = oracle_run(orc, inp, wl.n_steps)
    assert_same(got, want, key)


# ---------------------------------------------------------------------------
# shapes, thresholds, ranges, padding
# ---------------------------------------------------------------------------
SWEEP = [
    # (W, R, route_mode, thr, sizes, T, ld_pad, step0)
    (4, 1, wk.ROUTE_MOD, 65536, [1, 2, 3, 64, 65, 256], 4, 0, 0),
    (4, 1, wk.ROUTE_MOD, 0, [7, 57, 64, 1, 200], 3, 5, 0xFFFFFFFE),
    (5, 3, wk.ROUTE_MOD, 32768, [33, 31, 32, 64, 128, 129, 255, 256, 1], 5, 3, 7),
    (8, 4, wk.ROUTE_MOD, 1, [32] * 20 + [17, 5], 2, 0, 0),
    (13, 17, wk.ROUTE_MOD, 65535, [100, 30, 30, 4, 60, 200], 3, 64, 100),
    (16, 16, wk.ROUTE_CDF, 19661, [64] * 9 + [63, 1], 8, 0, 0),
    (31, 2, wk.ROUTE_CDF, 32768, [256, 256, 10, 54, 256], 2, 1, 0),
    (32, 64, wk.ROUTE_CDF, 19661, [256] * 5 + [160], 6, 0, 3),
    (33, 1024, wk.ROUTE_CDF, 3277, [32, 64, 128, 256, 5, 32, 32, 17], 4, 7, 0),
    (48, 1000, wk.ROUTE_MOD, 40000, [128, 128, 64, 64, 32, 32, 3], 3, 0, 0),
    (63, 5, wk.ROUTE_MOD, 32768, [1] * 70 + [256], 2, 2, 0),
    (64, 1024, wk.ROUTE_CDF, 3277, [256, 1, 255, 129, 127, 64, 33], 5, 0, 12345),
    (64, 256, wk.ROUTE_MOD, 32768, [256] * 3, 16, 0, 0),
    # two lanes per session with W < 32, three chunks of steps
    (24, 32, wk.ROUTE_MOD, 30000, [256, 100, 64, 33, 256], 40, 3, 5),
    (32, 128, wk.ROUTE_CDF, 19661, [256] * 3 + [200, 17], 37, 0, 0),
]


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("case", range(len(SWEEP)))
def test_shape_sweep(orc, case, mode):
    W, R, rmode, thr, sizes, T, pad, step0 = SWEEP[case]
    N = sum(sizes)
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=rmode, decide_thr=thr,
                         cohort_sizes=sizes, n_steps=T, seed_key=case, ld=N + pad)
    say("sweep case %d mode=%s W=%d R=%d thr=%d N=%d T=%d" % (case, mode, W, R, thr, N, T))
    got = gpu_run_ranges(inp, T, MODES[mode], [(0, inp.n_cohorts)], step0=step0)
    want = oracle_run(orc, inp, T, step0=step0)
    assert_same(got, want, "sweep %d" % case)


@pytest.mark.parametrize("mode", sorted(MODES))
def test_partial_cohort_ranges(orc, mode):
    """Only the cohorts in [begin, end) are touched, including ranges that
    start or end inside a packed workgroup."""
    sizes = [32, 20, 12, 64, 200, 7, 7, 50, 256, 31, 33]
    inp = wk.make_custom(n_words=9, n_routes=6, route_mode=wk.ROUTE_MOD, decide_thr=30000,
                         cohort_sizes=sizes, n_steps=3, seed_key=77, ld=sum(sizes) + 11)
    for cb, ce in [(1, 2), (2, 5), (5, 9), (0, 11), (10, 11), (3, 3)]:
        say("range [%d,%d) mode=%s" % (cb, ce, mode))
        got = gpu_run_ranges(inp, 3, MODES[mode], [(cb, ce)], step0=9)
        want = oracle_run(orc, inp, 3, step0=9, cb=cb, ce=ce)
        assert_same(got, want, "range %d-%d" % (cb, ce))


@pytest.mark.parametrize("mode", sorted(MODES))
def test_chain_composes_on_gpu(orc, mode):
    """run(T1, step0) then run(T2, step0 + T1) equals run(T1 + T2, step0)."""
    inp = wk.make_custom(n_words=32, n_routes=64, route_mode=wk.ROUTE_CDF, decide_thr=19661,
                         cohort_sizes=[256, 100, 64, 32, 32], n_steps=9, seed_key=5)
    T1, T2 = 4, 5
    co = rc.Cohort.from_inputs(inp, max_steps=T1 + T2)
    try:
        b1 = co.buffers
        co.run_chain(11, T1, MODES[mode])
        ld = co.ld
        import torch
        second = rc.RcBuffers(co.t["state"].data_ptr(), co.t["outcome"].data_ptr(),
                              co.t["eff_sid"][T1:].data_ptr(), co.t["eff_tool"][T1:].data_ptr(),
                              co.t["eff_payload"][T1:].data_ptr(), co.t["n_taken"][T1:].data_ptr(), ld)
        rc.rc_cohort_run_chain(co.handle, second, 11 + T1, T2, MODES[mode], 0, co.n_cohorts)
        torch.cuda.synchronize()
        got = co.download(T1 + T2)
        del b1
    finally:
        co.close()
    want = oracle_run(orc, inp, T1 + T2, step0=11)
    assert_same(got, want, "composed")


def test_resident_matches_host_roundtrip_and_is_deterministic():
    inp = wk.make_inputs(wk.WORKLOADS["s100k"])
    outs = []
    for mode in (rc.RC_MODE_RESIDENT, rc.RC_MODE_RESIDENT, rc.RC_MODE_HOST_ROUNDTRIP):
        outs.append(gpu_run_ranges(inp, 16, mode, [(0, inp.n_cohorts)]))
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), ("resident run twice", k)
        assert np.array_equal(outs[0][k], outs[2][k]), ("resident vs host round trip", k)


def test_launch_and_copy_counts():
    inp = wk.make_inputs(wk.WORKLOADS["k64"])
    co = rc.Cohort.from_inputs(inp, max_steps=8)
    try:
        co.run_chain(0, 8, rc.RC_MODE_RESIDENT, 0, 1)
        assert co.last_counts() == (1, 0)
        co.run_chain(0, 8, rc.RC_MODE_HOST_ROUNDTRIP, 1, 2)
        launches, copies = co.last_counts()
        assert copies == 8 and 8 + 8 <= launches <= 8 * 3
        co.step(0, 2, 3)
        assert co.last_counts() == (1, 0)
    finally:
        co.close()


def test_invalid_buffers_rejected_untouched():
    import torch
    inp = wk.make_custom(n_words=8, n_routes=4, route_mode=wk.ROUTE_MOD, decide_thr=32768,
                         cohort_sizes=[64, 64], n_steps=2, seed_key=3)
    co = rc.Cohort.from_inputs(inp, max_steps=2)
    try:
        before = co.download(2)
        t = co.t
        cases = {
            "overlap": rc.RcBuffers(t["state"].data_ptr(), t["state"].data_ptr(), t["eff_sid"].data_ptr(),
                                    t["eff_tool"].data_ptr(), t["eff_payload"].data_ptr(),
                                    t["n_taken"].data_ptr(), co.ld),
            "ld_small": rc.RcBuffers(t["state"].data_ptr(), t["outcome"].data_ptr(), t["eff_sid"].data_ptr(),
                                     t["eff_tool"].data_ptr(), t["eff_payload"].data_ptr(),
                                     t["n_taken"].data_ptr(), co.ld - 1),
            "null": rc.RcBuffers(0, t["outcome"].data_ptr(), t["eff_sid"].data_ptr(),
                                 t["eff_tool"].data_ptr(), t["eff_payload"].data_ptr(),
                                 t["n_taken"].data_ptr(), co.ld),
        }
        host = np.zeros(8 * co.ld, dtype=np.uint32)
        cases["host_memory"] = rc.RcBuffers(host.ctypes.data, t["outcome"].data_ptr(), t["eff_sid"].data_ptr(),
                                            t["eff_tool"].data_ptr(), t["eff_payload"].data_ptr(),
                                            t["n_taken"].data_ptr(), co.ld)
        for name, b in cases.items():
            st = rc.rc_cohort_run_chain(co.handle, b, 0, 2, rc.RC_MODE_RESIDENT, 0, 2, check=False)
            assert st == rc.RC_E_INVALID, name
        # a chain longer than the effect buffers is rejected (extent check)
        st = rc.rc_cohort_run_chain(co.handle, co.buffers, 0, 10 ** 6, rc.RC_MODE_RESIDENT, 0, 2,
                                    check=False)
        assert st == rc.RC_E_INVALID
        assert rc.rc_cohort_run_chain(co.handle, co.buffers, 0, 2, 7, 0, 2, check=False) == rc.RC_E_INVALID
        assert rc.rc_cohort_run_chain(co.handle, co.buffers, 0, 2, 0, 1, 3, check=False) == rc.RC_E_INVALID
        torch.cuda.synchronize()
        after = co.download(2)
        for k in before:
            assert np.array_equal(before[k], after[k]), k
    finally:
        co.close()


def test_empty_calls_are_noops():
    """n_steps == 0 or an empty cohort range: RC_OK, no launch, no copy, and
    every buffer bit-unchanged, in both mechanisms, the floor and step()."""
    import torch
    inp = wk.make_custom(n_words=32, n_routes=64, route_mode=wk.ROUTE_CDF, decide_thr=19661,
                         cohort_sizes=[256, 100, 31, 256], n_steps=2, seed_key=21,
                         ld=643 + 9)
    co = rc.Cohort.from_inputs(inp, max_steps=2)
    try:
        before = co.download(2)
        bits = np.full((2, (co.ld + 31) // 32), 0xFFFFFFFF, dtype=np.uint32)
        C = co.n_cohorts
        for mode in (rc.RC_MODE_RESIDENT, rc.RC_MODE_HOST_ROUNDTRIP):
            for T, cb, ce in ((0, 0, C), (2, 2, 2), (2, C, C), (0, 1, 1)):
                assert co.run_chain(5, T, mode, cb, ce) == rc.RC_OK
                assert co.last_counts() == (0, 0), (mode, T, cb, ce)
        dbits = torch.from_numpy(bits.view(np.int32)).to(co.device)
        for T, cb, ce in ((0, 0, C), (2, 3, 3)):
            assert rc.rc_cohort_run_floor(co.handle, co.buffers, dbits.data_ptr(), T, cb,
                                          ce) == rc.RC_OK
            assert co.last_counts() == (0, 0)
        assert co.step(0, 1, 1) == rc.RC_OK
        assert co.last_counts() == (0, 0)
        torch.cuda.synchronize()
        after = co.download(2)
        for k in before:
            assert np.array_equal(before[k], after[k]), k
    finally:
        co.close()


def mod_route_inputs(W, T, seed_key):
    """W words with mod-R routes (R = 256) in 600 cohorts, sub-wavefront and
    multi-wavefront sizes mixed, so that a launch of all of them takes more
    workgroups than the device has CUs."""
    rng = np.random.Generator(np.random.PCG64(seed_key))
    sizes = [int(x) for x in rng.choice([256, 256, 256, 200, 129, 128, 64, 40, 32, 1], size=600)]
    return wk.make_custom(n_words=W, n_routes=256, route_mode=wk.ROUTE_MOD, decide_thr=32768,
                          cohort_sizes=sizes, n_steps=T, seed_key=seed_key, ld=sum(sizes) + 3)


@pytest.mark.parametrize("W,T", [(32, 16), (32, 32), (16, 8), (13, 20)])
@pytest.mark.parametrize("mode", sorted(MODES))
def test_both_full_image_kernels(orc, mode, W, T):
    """Mod-R routes: one launch of every cohort (more workgroups than CUs:
    the two-role split at W = 32, the one-lane chain at W <= 16) and the same
    cohorts in launches of 1 to 220 cohorts (the pipelined three-role split,
    4-step chunks)."""
    inp = mod_route_inputs(W, T, 71_000 + 64 * W + T)
    C = inp.n_cohorts
    co = rc.Cohort.from_inputs(inp, max_steps=T)
    try:
        grid = co.plan_info()[0]
    finally:
        co.close()
    say("both full-image kernels mode=%s W=%d C=%d workgroups=%d T=%d" % (mode, W, C, grid, T))
    assert grid > 256
    want = oracle_run(orc, inp, T, step0=11)
    whole = gpu_run_ranges(inp, T, MODES[mode], [(0, C)], step0=11)
    assert_same(whole, want, "one launch")
    cuts = [0, 1, 101, 300, 520, C]
    pieces = gpu_run_ranges(inp, T, MODES[mode], list(zip(cuts[:-1], cuts[1:])), step0=11)
    assert_same(pieces, want, "launches of 1 to 220 cohorts")


@pytest.mark.parametrize("mode", sorted(MODES))
def test_cdf_routes_pipelined_at_every_size(orc, mode):
    """W = 32, T = 32, CDF routes (the k256 shape): the pipelined split at
    every launch size -- one launch of 1,000 cohorts, and launches of 1, 100
    and 256."""
    wl = wk.WORKLOADS["k256"]
    inp = wk.make_inputs(wl, chunk=1)
    C, T = inp.n_cohorts, wl.n_steps
    say("both two-lane kernels mode=%s C=%d T=%d" % (mode, C, T))
    want = oracle_run(orc, inp, T, step0=3)
    whole = gpu_run_ranges(inp, T, MODES[mode], [(0, C)], step0=3)
    assert_same(whole, want, "one launch")
    cuts = [0, 1, 101, 357, 613, 869, C]
    pieces = gpu_run_ranges(inp, T, MODES[mode], list(zip(cuts[:-1], cuts[1:])), step0=3)
    assert_same(pieces, want, "launches of 1 to 256 cohorts")
