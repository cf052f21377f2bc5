"""The no-decision floor on the GPU against the oracle (needs an MI355X).

The floor replays a given decision sequence through the resident chain with
no predicate (Section 7 "Matched mechanisms", "No-decision floor").  Two
kinds of check, both bit-exact over whole output arrays:

* the decisions the oracle itself makes (recorded by the oracle) replayed
  through the GPU floor give exactly the oracle's chain outputs;
* arbitrary decision bitmaps give exactly the oracle floor's outputs.
"""
import sys

import numpy as np
import pytest
import torch

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


def assert_same(got, want, what=""):
    for k in KEYS:
        g, w = got[k], want[k]
        assert g.shape == w.shape, (what, k, g.shape, w.shape)
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)
            raise AssertionError("%s: %s differs at %d places, first %s: gpu %#x oracle %#x"
                                 % (what, k, len(bad), tuple(bad[0]), int(g[tuple(bad[0])]),
                                    int(w[tuple(bad[0])])))


def gpu_floor(inp, bits, n_steps, ranges):
    co = rc.Cohort.from_inputs(inp, max_steps=n_steps)
    try:
        for cb, ce in ranges:
            co.run_floor(bits, n_steps, cb, ce)
        assert co.last_counts() == (1, 0)
        return co.download(n_steps)
    finally:
        co.close()


def random_bits(n_steps, ld, p, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    dec = rng.random((n_steps, ld)) < p
    words = np.zeros((n_steps, (ld + 31) // 32), dtype=np.uint64)
    for b in range(32):
        col = dec[:, b::32]
        words[:, :col.shape[1]] |= col.astype(np.uint64) << np.uint64(b)
    return words.astype(np.uint32)


@pytest.mark.parametrize("key,n_inv", [("tiny", 1000), ("k64", 1000), ("k256", 120),
                                       ("s100k", None), ("s1m", None)])
def test_floor_replays_oracle_decisions(orc, key, n_inv):
    """Recorded oracle decisions through the GPU floor = the oracle's chain."""
    wl = wk.WORKLOADS[key]
    inp = wk.make_inputs(wl, chunk=0) if n_inv else wk.make_inputs(wl)
    T = wl.n_steps
    ce = n_inv if n_inv else inp.n_cohorts
    say("floor case %s N=%d C=%d T=%d" % (key, inp.n_sessions, ce, T))
    want = orc.run_inputs(inp, n_steps=T, cohort_begin=0, cohort_end=ce, record=True)
    ranges = [(c, c + 1) for c in range(n_inv)] if n_inv else [(0, inp.n_cohorts)]
    got = gpu_floor(inp, want["decisions"], T, ranges)
    assert_same(got, want, key)


FLOOR_SWEEP = [
    # (W, R, route_mode, sizes, T, ld_pad, p_taken)
    (4, 1, wk.ROUTE_MOD, [1, 2, 3, 64, 65, 256], 5, 0, 0.5),
    (8, 4, wk.ROUTE_MOD, [32] * 20 + [17, 5], 17, 3, 0.9),
    (16, 16, wk.ROUTE_CDF, [64] * 9 + [63, 1], 33, 0, 0.3),
    (13, 17, wk.ROUTE_MOD, [100, 30, 30, 4, 60, 200], 3, 64, 0.0),
    (32, 256, wk.ROUTE_MOD, [256] * 5 + [160], 17, 0, 0.5),
    (32, 64, wk.ROUTE_CDF, [256, 256, 10, 54, 256], 1, 1, 1.0),
    (48, 1000, wk.ROUTE_MOD, [128, 128, 64, 64, 32, 32, 3], 6, 0, 0.2),
    (64, 1024, wk.ROUTE_CDF, [256, 1, 255, 129, 127, 64, 33], 5, 7, 0.05),
    (64, 200, wk.ROUTE_MOD, [256] * 3 + [31], 9, 0, 0.6),
    # two lanes per session: beyond the two chunks whose decisions are
    # loaded up front, and W < 32
    (32, 128, wk.ROUTE_CDF, [256] * 3 + [200, 17], 40, 0, 0.4),
    (20, 8, wk.ROUTE_MOD, [256, 40, 90], 33, 5, 0.7),
]


@pytest.mark.parametrize("case", range(len(FLOOR_SWEEP)))
def test_floor_arbitrary_decisions(orc, case):
    """Random decision bitmaps: GPU floor = oracle floor, whole launch and
    ragged cohort ranges."""
    W, R, rmode, sizes, T, pad, p = FLOOR_SWEEP[case]
    N = sum(sizes)
    inp = wk.make_custom(n_words=W, n_routes=R, route_mode=rmode, decide_thr=32768,
                         cohort_sizes=sizes, n_steps=T, seed_key=500 + case, ld=N + pad)
    bits = random_bits(T, inp.ld, p, 600 + case)
    C = inp.n_cohorts
    say("floor sweep %d W=%d R=%d N=%d T=%d p=%.2f" % (case, W, R, N, T, p))
    want = orc.run_inputs(inp, n_steps=T, decisions=bits)
    got = gpu_floor(inp, bits, T, [(0, C)])
    assert_same(got, want, "floor sweep %d" % case)
    # the same cohorts in ragged ranges, one call each, in a shuffled order
    cuts = sorted(set([0, C] + [int(x) for x in np.linspace(0, C, 4)[1:-1]]))
    ranges = [(cuts[i], cuts[i + 1]) for i in range(len(cuts) - 1)][::-1]
    got = gpu_floor(inp, bits, T, ranges)
    assert_same(got, want, "floor sweep %d, ranges %s" % (case, ranges))


def test_floor_invalid_arguments_touch_nothing():
    inp = wk.make_custom(n_words=8, n_routes=4, route_mode=wk.ROUTE_MOD, decide_thr=32768,
                         cohort_sizes=[64, 32], n_steps=2, seed_key=7, ld=100)
    co = rc.Cohort.from_inputs(inp, max_steps=2)
    try:
        before = co.download(2)
        # (a bitmap shorter than its extent is caught only when the extent
        # leaves its allocation; torch's caching allocator sub-allocates
        # larger segments, so that case is not constructed here)
        bits = torch.zeros((2, (inp.ld + 31) // 32), dtype=torch.int32, device="cuda")
        host = np.zeros((2, 4), dtype=np.uint32)
        cases = [
            ("null decisions", 0, 2, 0, 2),
            ("decisions overlap the state", co.t["state"].data_ptr(), 2, 0, 2),
            ("decisions overlap the effect log", co.t["eff_tool"].data_ptr(), 2, 0, 2),
            ("decisions in host memory", host.ctypes.data, 2, 0, 2),
            ("bad cohort range", bits.data_ptr(), 2, 1, 3),
        ]
        for what, ptr, T, cb, ce in cases:
            st = rc.rc_cohort_run_floor(co.handle, co.buffers, ptr, T, cb, ce, check=False)
            assert st == rc.RC_E_INVALID, (what, rc.rc_status_string(st))
        after = co.download(2)
        for k in KEYS:
            assert np.array_equal(before[k], after[k]), k
    finally:
        co.close()


@pytest.mark.parametrize("W", [32, 16])
def test_floor_both_full_image_kernels(orc, W):
    """T = 32, mod-R routes, with the oracle's recorded decisions: one launch
    of 600 cohorts (more workgroups than CUs: the two-role split at W = 32,
    the one-lane chain at W = 16) and launches of at most 256 cohorts (the
    pipelined three-role split) reproduce the oracle's chain."""
    T = 32
    rng = np.random.Generator(np.random.PCG64(72_000 + W))
    sizes = [int(x) for x in rng.choice([256, 256, 256, 200, 129, 128, 64, 40, 32, 1], size=600)]
    inp = wk.make_custom(n_words=W, n_routes=256, route_mode=wk.ROUTE_MOD, decide_thr=32768,
                         cohort_sizes=sizes, n_steps=T, seed_key=72_000 + W, ld=sum(sizes) + 3)
    C = inp.n_cohorts
    say("floor, both full-image kernels: W=%d C=%d T=%d" % (W, C, T))
    want = orc.run_inputs(inp, n_steps=T, record=True)
    whole = gpu_floor(inp, want["decisions"], T, [(0, C)])
    assert_same(whole, want, "one launch")
    cuts = [0, 256, 257, 400, C]
    pieces = gpu_floor(inp, want["decisions"], T, list(zip(cuts[:-1], cuts[1:])))
    assert_same(pieces, want, "launches of at most 256 cohorts")
